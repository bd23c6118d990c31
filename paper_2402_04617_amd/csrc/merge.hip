// Log-sum-exp merge of partial attentions over disjoint key parts:
// LSE = log sum_s exp(lse_s), O = sum_s exp(lse_s - LSE) O_s.  The parts together
// are the single softmax over Concat(C, X) of Section 3.1.
//
// One thread per (row, 16 bytes of partial row): 8 dims of a scaled-fp16 partial
// (bfloat16 inputs; value * 2^exp[row] restores the row) or 4 dims of a float32
// one.  Parts are taken CH at a time (CH = the part count when it is at most 8,
// so the usual launch issues exactly its loads, all before the first use);
// longer part lists run in chunks joined by a running maximum, the indices of a
// short last chunk clamped to the last part and its surplus weights zero.
#include "launch.h"

namespace infllm {
namespace {

template <typename T, bool HALF, int CH>
__global__ void __launch_bounds__(256) merge_kernel(MergeArgs a) {
  constexpr int DPT = HALF ? 8 : 4;  // dims per thread
  const int tpr = a.head_dim / DPT;
  const int rows_per_wg = 256 / tpr;
  // Workgroups in the attention's XCD order (reversed, consecutive ids on one
  // XCD): where a kv head's parts were written by the workgroups of one XCD, the
  // rows of that kv head are merged on the same XCD and read its L2.
  const int wg = (int)gridDim.x - 1 - xcd_logical_block(blockIdx.x, gridDim.x);
  const int row = wg * rows_per_wg + threadIdx.x / tpr;
  const int c = threadIdx.x % tpr;
  if (row >= a.rows) return;
  float M = -__builtin_inff(), tot = 0.f;
  float acc[DPT];
#pragma unroll
  for (int e = 0; e < DPT; ++e) acc[e] = 0.f;
  for (int s0 = 0; s0 < a.parts; s0 += CH) {
    float l[CH], o[CH][DPT];
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const int64_t pr = (int64_t)min(s0 + j, a.parts - 1) * a.rows + row;
      l[j] = a.part_lse[pr];
      if constexpr (HALF) {
        const uint4 w = *(const uint4*)((const uint16_t*)a.part_o + pr * a.head_dim + DPT * c);
        const float sc = exp2_int(a.part_exp[pr]);
        const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          o[j][2 * q] = f16_lo(ww[q]) * sc;
          o[j][2 * q + 1] = f16_hi(ww[q]) * sc;
        }
      } else {
        const float4 w = *(const float4*)((const float*)a.part_o + pr * a.head_dim + DPT * c);
        o[j][0] = w.x;
        o[j][1] = w.y;
        o[j][2] = w.z;
        o[j][3] = w.w;
      }
    }
    float mc = -__builtin_inff();
#pragma unroll
    for (int j = 0; j < CH; ++j)
      if (s0 + j < a.parts) mc = fmaxf(mc, l[j]);
    const float m_new = fmaxf(M, mc);
    if (m_new == -__builtin_inff()) continue;  // nothing visible yet
    const float r = M == -__builtin_inff() ? 0.f : expf(M - m_new);
    tot *= r;
#pragma unroll
    for (int e = 0; e < DPT; ++e) acc[e] *= r;
#pragma unroll
    for (int j = 0; j < CH; ++j) {
      const float w = (s0 + j < a.parts && l[j] != -__builtin_inff()) ? expf(l[j] - m_new) : 0.f;
      tot += w;
#pragma unroll
      for (int e = 0; e < DPT; ++e) acc[e] += w * o[j][e];
    }
    M = m_new;
  }
  const float inv = tot > 0.f ? 1.f / tot : 0.f;
  const int bh = row / a.n_q, i = row - bh * a.n_q;
  T* op = (T*)a.out + (int64_t)bh * a.out_head_stride + (int64_t)i * a.head_dim + DPT * c;
  if constexpr (sizeof(T) == 2) {
    uint32_t w[DPT / 2];
#pragma unroll
    for (int q = 0; q < DPT / 2; ++q)
      w[q] = (uint32_t)f32_to_bf16(acc[2 * q] * inv) | ((uint32_t)f32_to_bf16(acc[2 * q + 1] * inv) << 16);
    if constexpr (DPT == 8) *(uint4*)op = make_uint4(w[0], w[1], w[2], w[3]);
    else *(uint2*)op = make_uint2(w[0], w[1]);
  } else {
#pragma unroll
    for (int e = 0; e < DPT; ++e) op[e] = acc[e] * inv;
  }
  if (a.lse != nullptr && c == 0) a.lse[row] = tot > 0.f ? M + logf(tot) : -__builtin_inff();
}

template <typename T, bool HALF>
hipError_t launch_merge_t(const MergeArgs& a, hipStream_t s) {
  constexpr int DPT = HALF ? 8 : 4;
  const int rows_per_wg = 256 / (a.head_dim / DPT);
  const dim3 grid((a.rows + rows_per_wg - 1) / rows_per_wg), block(256);
  switch (a.parts) {
    case 2: hipLaunchKernelGGL((merge_kernel<T, HALF, 2>), grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL((merge_kernel<T, HALF, 3>), grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL((merge_kernel<T, HALF, 4>), grid, block, 0, s, a); break;
    default: hipLaunchKernelGGL((merge_kernel<T, HALF, 8>), grid, block, 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, hipStream_t s) {
  if (a.rows == 0) return hipSuccess;
  return a.bf16 ? launch_merge_t<bf16_t, true>(a, s) : launch_merge_t<float, false>(a, s);
}

}  // namespace infllm
