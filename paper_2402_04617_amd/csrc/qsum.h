// Block-level sum of a chunk's queries over a kv head's query group, shared by
// the scoring kernels and the append launch (Mean Repr path).  Rows of the
// group are (head, i) pairs, head-major; part `part` of `parts` sums an equal
// share of them in a fixed order, so the partial sums are deterministic.
#pragma once

#include "launch.h"

namespace infllm {

constexpr int kQsumThreads = 256;  // threads of the scoring kernels' query-sum blocks

// NT: the block's thread count (all of them take part).
template <typename T, int NT = kQsumThreads>
struct QsumSmem {
  float red[NT * (16 / sizeof(T))];
};

template <typename T, int NT = kQsumThreads>
__device__ __forceinline__ void qsum_block(const T* __restrict__ q, int64_t q_head_stride, int n_q_heads,
                                           int n_kv_heads, int head_dim, int n_q, int part, int parts, int bg,
                                           float* __restrict__ qbar_parts, QsumSmem<T, NT>& sm) {
  constexpr int kVec = 16 / sizeof(T);
  const int b = bg / n_kv_heads, g = bg - b * n_kv_heads;
  const int G = n_q_heads / n_kv_heads;
  const int rows = G * n_q;
  const int per = (rows + parts - 1) / parts;
  const int r0 = min(rows, part * per), r1 = min(rows, r0 + per);
  const int lanes_per_row = head_dim / kVec;
  const int rgroups = NT / lanes_per_row;
  const int c = threadIdx.x % lanes_per_row;
  const int rg = threadIdx.x / lanes_per_row;

  float acc[kVec];
#pragma unroll
  for (int e = 0; e < kVec; ++e) acc[e] = 0.f;
  // kBatch rows per thread are loaded before the first add (one memory round
  // trip per batch); rows past the part add zeros, so each thread sums its rows
  // in the same order whatever the batching
  constexpr int kBatch = 8;
  for (int r = r0 + rg; r < r1; r += kBatch * rgroups) {
    uint4 raw[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int rr = r + u * rgroups;
      raw[u] = make_uint4(0u, 0u, 0u, 0u);
      if (rr < r1) {
        const int hl = rr / n_q, i = rr - hl * n_q;
        const T* row = q + (int64_t)(b * n_q_heads + g * G + hl) * q_head_stride + (int64_t)i * head_dim;
        raw[u] = *(const uint4*)(row + c * kVec);
      }
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const T* vals = (const T*)&raw[u];
#pragma unroll
      for (int e = 0; e < kVec; ++e) acc[e] += Elem<T>::load(vals + e);
    }
  }
#pragma unroll
  for (int e = 0; e < kVec; ++e) sm.red[rg * head_dim + c * kVec + e] = acc[e];
  __syncthreads();
  for (int d = threadIdx.x; d < head_dim; d += NT) {
    float s = 0.f;
    for (int j = 0; j < rgroups; ++j) s += sm.red[j * head_dim + d];
    qbar_parts[((int64_t)bg * parts + part) * head_dim + d] = s;
  }
}

}  // namespace infllm
