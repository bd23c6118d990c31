// Log-sum-exp merge of partial attentions over disjoint key parts:
// LSE = log sum_s exp(lse_s), O = sum_s exp(lse_s - LSE) O_s.  The parts together
// are the single softmax over Concat(C, X) of Section 3.1.
#include "launch.h"

namespace infllm {
namespace {

template <typename T>
__global__ void __launch_bounds__(256) merge_kernel(MergeArgs a) {
  const int tpr = a.head_dim / 4;
  const int rows_per_wg = 256 / tpr;
  const int row = blockIdx.x * rows_per_wg + threadIdx.x / tpr;
  const int c = threadIdx.x % tpr;
  if (row >= a.rows) return;
  float M = -__builtin_inff();
  for (int s = 0; s < a.parts; ++s) M = fmaxf(M, a.part_lse[(int64_t)s * a.rows + row]);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float tot = 0.f;
  if (M != -__builtin_inff()) {
    for (int s = 0; s < a.parts; ++s) {
      const float w = expf(a.part_lse[(int64_t)s * a.rows + row] - M);
      const float4 o = *(const float4*)(a.part_o + ((int64_t)s * a.rows + row) * a.head_dim + 4 * c);
      acc.x += w * o.x;
      acc.y += w * o.y;
      acc.z += w * o.z;
      acc.w += w * o.w;
      tot += w;
    }
  }
  const float inv = tot > 0.f ? 1.f / tot : 0.f;
  const int bh = row / a.n_q, i = row - bh * a.n_q;
  T* op = (T*)a.out + (int64_t)bh * a.out_head_stride + (int64_t)i * a.head_dim + 4 * c;
  Elem<T>::store(op + 0, acc.x * inv);
  Elem<T>::store(op + 1, acc.y * inv);
  Elem<T>::store(op + 2, acc.z * inv);
  Elem<T>::store(op + 3, acc.w * inv);
  if (a.lse != nullptr && c == 0) a.lse[row] = tot > 0.f ? M + logf(tot) : -__builtin_inff();
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, hipStream_t s) {
  if (a.rows == 0) return hipSuccess;
  const int rows_per_wg = 256 / (a.head_dim / 4);
  dim3 grid((a.rows + rows_per_wg - 1) / rows_per_wg);
  if (a.bf16)
    hipLaunchKernelGGL(merge_kernel<bf16_t>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(merge_kernel<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace infllm
