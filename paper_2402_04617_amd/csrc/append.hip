// Append of the current tokens: K/V into the token-ordered store, and the
// running group-query sum into the float64 ring that unit construction reads.
//
// The representative score of Section 3.2 needs, for every token m, the window
// sum W_m = sum_{j=1..l_L} sum_{h in group} q^h_{m+j}.  Keeping the running sum
// Pi_t = sum_{p<=t} sum_h q^h_p lets unit construction form W_m as one difference
// of two ring slots, so its cost does not grow with l_L.  float64 keeps the
// difference of two large running sums exact to ~1e-16 relative.
#include "launch.h"

namespace infllm {
namespace {

// 16-byte vector copy of the chunk's K (or V) rows into the store.
__global__ void copy_rows_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                 int64_t vec_per_head, int64_t src_head_stride_vec,
                                 int64_t dst_head_stride_vec, int64_t dst_offset_vec,
                                 int64_t total_vec) {
  int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= total_vec) return;
  int64_t head = e / vec_per_head;
  int64_t r = e - head * vec_per_head;
  dst[head * dst_head_stride_vec + dst_offset_vec + r] = src[head * src_head_stride_vec + r];
}

// One workgroup per (sequence*kv head, 32-dim slice); 8 segments of the chunk
// are summed in parallel, then scanned, then re-walked to write every slot.
template <typename T>
__global__ void __launch_bounds__(256) qprefix_kernel(const T* __restrict__ q, int64_t q_head_stride,
                                                      int n_q_heads, int n_kv_heads, int head_dim,
                                                      int n_q, int64_t past_len,
                                                      double* __restrict__ qprefix, int ring) {
  constexpr int kSegs = 8;
  const int bg = blockIdx.x;
  const int b = bg / n_kv_heads, g = bg - b * n_kv_heads;
  const int lane = threadIdx.x & 31;
  const int seg = threadIdx.x >> 5;
  const int d = blockIdx.y * 32 + lane;
  const int G = n_q_heads / n_kv_heads;
  const int seg_len = (n_q + kSegs - 1) / kSegs;
  const int i0 = min(n_q, seg * seg_len), i1 = min(n_q, i0 + seg_len);
  const T* qb = q + (int64_t)(b * n_q_heads + g * G) * q_head_stride + d;

  double acc = 0.0;
  for (int i = i0; i < i1; ++i) {
    double s = 0.0;
    for (int h = 0; h < G; ++h) s += (double)Elem<T>::load(qb + h * q_head_stride + (int64_t)i * head_dim);
    acc += s;
  }
  __shared__ double seg_sum[kSegs][32];
  seg_sum[seg][lane] = acc;
  __syncthreads();

  double* ring_bg = qprefix + (int64_t)bg * ring * head_dim;
  double run = 0.0;
  if (past_len > 0) run = ring_bg[((past_len - 1) % ring) * head_dim + d];
  for (int s = 0; s < seg; ++s) run += seg_sum[s][lane];
  // Every thread has read the base slot before any slot is written (the new
  // slots never alias it because ring > n_q).
  __syncthreads();
  for (int i = i0; i < i1; ++i) {
    double s = 0.0;
    for (int h = 0; h < G; ++h) s += (double)Elem<T>::load(qb + h * q_head_stride + (int64_t)i * head_dim);
    run += s;
    ring_bg[((past_len + i) % ring) * head_dim + d] = run;
  }
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, hipStream_t s) {
  if (a.n_q == 0) return hipSuccess;
  const int esize = a.bf16 ? 2 : 4;
  const int vec = 16 / esize;
  if (a.k_src != nullptr) {
    int64_t vec_per_head = (int64_t)a.n_q * a.head_dim / vec;
    int64_t heads = (int64_t)a.batch * a.n_kv_heads;
    int64_t total = vec_per_head * heads;
    int64_t src_stride = a.kv_head_stride / vec;
    int64_t dst_stride = a.capacity * a.head_dim / vec;
    int64_t dst_off = a.past_len * a.head_dim / vec;
    dim3 grid((unsigned)((total + 255) / 256));
    hipLaunchKernelGGL(copy_rows_kernel, grid, dim3(256), 0, s, (const uint4*)a.k_src, (uint4*)a.k_store,
                       vec_per_head, src_stride, dst_stride, dst_off, total);
    hipLaunchKernelGGL(copy_rows_kernel, grid, dim3(256), 0, s, (const uint4*)a.v_src, (uint4*)a.v_store,
                       vec_per_head, src_stride, dst_stride, dst_off, total);
  }
  dim3 grid(a.batch * a.n_kv_heads, a.head_dim / 32);
  if (a.bf16)
    hipLaunchKernelGGL(qprefix_kernel<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)a.q, a.q_head_stride,
                       a.n_q_heads, a.n_kv_heads, a.head_dim, a.n_q, a.past_len, a.qprefix, a.ring);
  else
    hipLaunchKernelGGL(qprefix_kernel<float>, grid, dim3(256), 0, s, (const float*)a.q, a.q_head_stride,
                       a.n_q_heads, a.n_kv_heads, a.head_dim, a.n_q, a.past_len, a.qprefix, a.ring);
  return hipGetLastError();
}

}  // namespace infllm
