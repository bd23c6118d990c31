// Memory-unit construction (Section 3.2, "Block-Level Memory Units") as a
// block-level device routine, shared by the standalone unit-construction kernel
// and the fused append launch of the whole-step path.
//
// One block per (unit, sequence*kv head).  Token m of the unit has
// l_L*G*r_m = k_m . W_m, W_m = sum_{h in group} sum_{j=1..l_L} q^h_{m+j}, which the
// append scan already stored as D/kRpartDims float64 partial sums (rpart); here they are
// added in slice order (one token per thread, all loads in flight together).
// The r_k tokens of largest r_m (ties: lower position) become R(B): each token's
// rank under that strict order is counted against all others in LDS, split over
// several threads per token, and a ballot scan gives the ascending slot.  The
// unit stores the offsets and the sum of its representative keys (what unit
// scoring streams).
#pragma once

#include "launch.h"

namespace infllm {

constexpr int kMaxBlock = 256;        // largest l_bs
constexpr int kMaxSumElems = 2048;    // staged representative-key elements

// LDS of one unit-construction block.
struct BuildSmem {
  __attribute__((aligned(16))) double r[kMaxBlock];
  int chosen[kMaxBlock];
  int wave_cnt[16];
  float rk[kMaxSumElems];
};

template <typename T, int D, int NT>
__device__ __forceinline__ void build_one_unit(const BuildArgs& a, int unit, int unit_local, int bg,
                                               BuildSmem& sm) {
  static_assert(NT % 64 == 0 && NT >= 256 && NT <= 1024, "block size");
  constexpr int SLICES = D / kRpartDims;
  const int lbs = a.block_size;
  const int tid = threadIdx.x;
  const int64_t m0 = (int64_t)a.n_init + (int64_t)unit * lbs;
  const T* kb = (const T*)a.k_store + ((int64_t)bg * a.capacity) * D;
  const double* rp = a.rpart + (int64_t)bg * SLICES * a.ring;
  // ring slot of the unit's first token; the ring holds more than l_bs slots, so
  // stepping by t < l_bs wraps at most once
  const int slot0 = (int)(m0 % a.ring);

  double* r = sm.r;
  int* chosen = sm.chosen;
  int* wave_cnt = sm.wave_cnt;

  for (int t = tid; t < lbs; t += NT) {
    int st = slot0 + t;
    st -= (st >= a.ring) ? a.ring : 0;
    double x[SLICES];
#pragma unroll
    for (int s = 0; s < SLICES; ++s) x[s] = rp[(int64_t)s * a.ring + st];
    double acc = 0.0;
#pragma unroll
    for (int s = 0; s < SLICES; ++s) acc += x[s];
    r[t] = (acc != acc) ? -__builtin_inf() : acc;  // NaN ranks lowest
  }
  __syncthreads();

  // Rank under the strict order (larger r first, then lower offset); the r_k
  // tokens of rank < r_k are the representatives.  TPT adjacent threads share a
  // token, each counting against every TPT-th other token.
  int tpt = 1;
  while (tpt < 8 && tpt * 2 * lbs <= NT) tpt *= 2;
  const int t = tid / tpt, sub = tid - t * tpt;
  int rank = 0;
  if (t < lbs) {
    const double rt = r[t];
    int u = sub;
    for (; u + 3 * tpt < lbs; u += 4 * tpt) {
      const double x0 = r[u], x1 = r[u + tpt], x2 = r[u + 2 * tpt], x3 = r[u + 3 * tpt];
      rank += (x0 > rt) || (x0 == rt && u < t);
      rank += (x1 > rt) || (x1 == rt && u + tpt < t);
      rank += (x2 > rt) || (x2 == rt && u + 2 * tpt < t);
      rank += (x3 > rt) || (x3 == rt && u + 3 * tpt < t);
    }
    for (; u < lbs; u += tpt) {
      const double ru = r[u];
      rank += (ru > rt) || (ru == rt && u < t);
    }
  }
  for (int o = 1; o < tpt; o <<= 1) rank += __shfl_xor(rank, o);
  const bool sel = t < lbs && sub == 0 && rank < a.n_repr;
  const int lane = tid & 63, wave = tid >> 6;
  const unsigned long long mask = __ballot(sel);
  if (lane == 0) wave_cnt[wave] = __popcll(mask);
  __syncthreads();
  if (sel) {
    int slot = __popcll(mask & ((1ull << lane) - 1ull));
    for (int w = 0; w < wave; ++w) slot += wave_cnt[w];
    chosen[slot] = t;
    a.repr_idx[((int64_t)bg * a.max_units + unit) * a.n_repr + slot] = t;
  }
  __syncthreads();

  // Sum of the representative keys, in ascending position order, float32:
  // one load per (representative, dim) thread, then a fixed-order sum in LDS.
  float* rk = sm.rk;
  const int nrep_load = min(a.n_repr, kMaxSumElems / D);
  for (int e = tid; e < nrep_load * D; e += NT) {
    const int j = e / D, d = e - j * D;
    rk[e] = Elem<T>::load(kb + (m0 + chosen[j]) * D + d);
  }
  __syncthreads();
  for (int d = tid; d < D; d += NT) {
    float s = 0.f;
    for (int j = 0; j < nrep_load; ++j) s += rk[j * D + d];
    for (int j = nrep_load; j < a.n_repr; ++j) s += Elem<T>::load(kb + (m0 + chosen[j]) * D + d);
    a.unit_ksum[(((int64_t)bg * (D / 4) + d / 4) * a.max_units + unit) * 4 + (d & 3)] = s;
  }
  if (a.repr_score != nullptr) {
    const int G = a.n_q_heads / a.n_kv_heads;
    const double norm = 1.0 / ((double)a.n_local * (double)G);
    for (int u = tid; u < lbs; u += NT)
      a.repr_score[((int64_t)bg * a.n_new + unit_local) * lbs + u] = r[u] * norm;
  }
}

// Mean representation (the paper's "Mean Repr" alternative, Section 4): the
// unit is scored by the mean of all its l_bs keys.  Each key row is read as
// 16-byte pieces by LPK adjacent threads; KG groups of them take interleaved
// rows, and the groups' partial sums are added in a fixed order.
template <typename T, int D, int NT>
__device__ __forceinline__ void mean_one_unit(const BuildArgs& a, int unit, int bg, BuildSmem& sm) {
  constexpr int VEC = 16 / (int)sizeof(T);  // elements per 16-byte piece
  constexpr int LPK = D / VEC;              // threads per key row
  constexpr int KG = (NT / LPK) < (kMaxSumElems / D) ? (NT / LPK) : (kMaxSumElems / D);
  const int lbs = a.block_size;
  const int64_t m0 = (int64_t)a.n_init + (int64_t)unit * lbs;
  const T* kb = (const T*)a.k_store + ((int64_t)bg * a.capacity + m0) * D;
  const int c = threadIdx.x % LPK, grp = threadIdx.x / LPK;
  if (grp < KG) {
    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
#pragma unroll 4
    for (int j = grp; j < lbs; j += KG) {
      const uint4 raw = *(const uint4*)(kb + (int64_t)j * D + c * VEC);
      const T* vals = (const T*)&raw;
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] += Elem<T>::load(vals + e);
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) sm.rk[grp * D + c * VEC + e] = acc[e];
  }
  __syncthreads();
  for (int d = threadIdx.x; d < D; d += NT) {
    float s = 0.f;
#pragma unroll
    for (int g = 0; g < KG; ++g) s += sm.rk[g * D + d];
    a.unit_ksum[(((int64_t)bg * (D / 4) + d / 4) * a.max_units + unit) * 4 + (d & 3)] = s / (float)lbs;
  }
}

// Unit `unit_local` of the units this (sequence, kv head) builds, in either
// representation.  In a variable-length batch each sequence has its own range;
// blocks past a sequence's count return at once (before any barrier).
template <typename T, int D, int NT>
__device__ __forceinline__ void construct_unit(const BuildArgs& a, int unit_local, int bg, BuildSmem& sm) {
  int first = a.first_unit, count = a.n_new;
  if (a.var_on) {
    const int b = bg / a.n_kv_heads;
    first = a.var_first[b];
    count = a.var_count[b];
  }
  if (unit_local >= count) return;
  if (a.mean_repr) mean_one_unit<T, D, NT>(a, first + unit_local, bg, sm);
  else build_one_unit<T, D, NT>(a, first + unit_local, unit_local, bg, sm);
}

}  // namespace infllm
