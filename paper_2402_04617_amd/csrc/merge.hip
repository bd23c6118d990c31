// Log-sum-exp merge of partial attentions over disjoint key parts:
// LSE = log sum_s exp(lse_s), O = sum_s exp(lse_s - LSE) O_s.  The parts together
// are the single softmax over Concat(C, X) of Section 3.1.
//
// One thread per (row, 4 dims).  Parts are taken kChunk at a time with every
// load of the chunk issued before the first use (indices clamped to the last
// part, surplus weights zero), and chunks are joined with a running maximum, so
// any part count is exact and the usual one-chunk case waits on memory once.
// Partial rows are float32 for float32 inputs and scaled fp16 for bfloat16
// inputs (value * 2^exp[row] restores the row).
#include "launch.h"

namespace infllm {
namespace {

constexpr int kChunk = 8;

template <typename T, bool HALF>
__global__ void __launch_bounds__(256) merge_kernel(MergeArgs a) {
  const int tpr = a.head_dim / 4;
  const int rows_per_wg = 256 / tpr;
  const int row = blockIdx.x * rows_per_wg + threadIdx.x / tpr;
  const int c = threadIdx.x % tpr;
  if (row >= a.rows) return;
  float M = -__builtin_inff(), tot = 0.f;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < a.parts; s0 += kChunk) {
    float l[kChunk], o[kChunk][4];
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
      const int64_t pr = (int64_t)min(s0 + j, a.parts - 1) * a.rows + row;
      l[j] = a.part_lse[pr];
      if constexpr (HALF) {
        const uint2 w = *(const uint2*)((const uint16_t*)a.part_o + pr * a.head_dim + 4 * c);
        const float sc = exp2_int(a.part_exp[pr]);
        o[j][0] = f16_lo(w.x) * sc;
        o[j][1] = f16_hi(w.x) * sc;
        o[j][2] = f16_lo(w.y) * sc;
        o[j][3] = f16_hi(w.y) * sc;
      } else {
        const float4 w = *(const float4*)((const float*)a.part_o + pr * a.head_dim + 4 * c);
        o[j][0] = w.x;
        o[j][1] = w.y;
        o[j][2] = w.z;
        o[j][3] = w.w;
      }
    }
    float mc = -__builtin_inff();
#pragma unroll
    for (int j = 0; j < kChunk; ++j)
      if (s0 + j < a.parts) mc = fmaxf(mc, l[j]);
    const float m_new = fmaxf(M, mc);
    if (m_new == -__builtin_inff()) continue;  // nothing visible yet
    const float r = M == -__builtin_inff() ? 0.f : expf(M - m_new);
    tot *= r;
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] *= r;
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
      const float w = (s0 + j < a.parts && l[j] != -__builtin_inff()) ? expf(l[j] - m_new) : 0.f;
      tot += w;
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] += w * o[j][e];
    }
    M = m_new;
  }
  const float inv = tot > 0.f ? 1.f / tot : 0.f;
  const int bh = row / a.n_q, i = row - bh * a.n_q;
  T* op = (T*)a.out + (int64_t)bh * a.out_head_stride + (int64_t)i * a.head_dim + 4 * c;
  if constexpr (sizeof(T) == 2) {
    uint2 w;
    w.x = (uint32_t)f32_to_bf16(acc[0] * inv) | ((uint32_t)f32_to_bf16(acc[1] * inv) << 16);
    w.y = (uint32_t)f32_to_bf16(acc[2] * inv) | ((uint32_t)f32_to_bf16(acc[3] * inv) << 16);
    *(uint2*)op = w;
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) op[e] = acc[e] * inv;
  }
  if (a.lse != nullptr && c == 0) a.lse[row] = tot > 0.f ? M + logf(tot) : -__builtin_inff();
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, hipStream_t s) {
  if (a.rows == 0) return hipSuccess;
  const int rows_per_wg = 256 / (a.head_dim / 4);
  dim3 grid((a.rows + rows_per_wg - 1) / rows_per_wg);
  if (a.bf16)
    hipLaunchKernelGGL((merge_kernel<bf16_t, true>), grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((merge_kernel<float, false>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace infllm
