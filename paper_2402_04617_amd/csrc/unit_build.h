// Memory-unit construction (Section 3.2, "Block-Level Memory Units") as a
// block-level device routine, shared by the standalone unit-construction kernel
// and the fused append launch of the whole-step path.
//
// One block per (unit, sequence*kv head).  Each token m of the unit gets
// r_m = k_m . W_m with W_m = Pi_{m+l_L} - Pi_m read from the float64 running-sum
// ring (slot t holds the group's query sum through position t), which equals
// sum_{h in group} sum_{j=1..l_L} q^h_{m+j} . k_m.  Eight threads share a token
// (an eighth of the head dim each), all loads issued before any arithmetic.  The
// r_k tokens of largest r_m (ties: lower position) become R(B): each token's rank
// under that strict order is counted against all others in LDS, and a ballot
// scan gives the ascending slot.  The unit stores the offsets and the sum of its
// representative keys (what unit scoring streams).
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
__device__ __forceinline__ void build_one_unit(const BuildArgs& a, int unit_local, int bg, BuildSmem& sm) {
  constexpr int SL = D / 8;  // dims per thread: 8 threads per token
  static_assert(NT % 64 == 0 && NT >= 256 && NT <= 1024, "block size");
  constexpr int TPP = NT / 8;  // tokens per pass (8 threads per token)
  const int unit = a.first_unit + unit_local;
  const int lbs = a.block_size;
  const int tid = threadIdx.x;
  const int64_t m0 = (int64_t)a.n_init + (int64_t)unit * lbs;
  const T* kb = (const T*)a.k_store + ((int64_t)bg * a.capacity) * D;
  const double* ring = a.qprefix + (int64_t)bg * a.ring * D;
  // ring slots of the unit's first token and of its window end; the ring holds
  // at least l_bs + l_L slots, so stepping by t < l_bs wraps at most once
  const int slot_lo0 = (int)(m0 % a.ring);
  const int slot_hi0 = (int)((m0 + a.n_local) % a.ring);

  double* r = sm.r;
  int* chosen = sm.chosen;
  int* wave_cnt = sm.wave_cnt;

  const int sl = tid & 7;
  for (int t = tid >> 3; t < lbs; t += TPP) {
    int slo = slot_lo0 + t, shi = slot_hi0 + t;
    slo -= (slo >= a.ring) ? a.ring : 0;
    shi -= (shi >= a.ring) ? a.ring : 0;
    const double* hi = ring + (int64_t)shi * D + sl * SL;
    const double* lo = ring + (int64_t)slo * D + sl * SL;
    const T* km = kb + (m0 + t) * D + sl * SL;
    float kv[SL];
    double2 h2[SL / 2], l2[SL / 2];
#pragma unroll
    for (int e = 0; e < SL; e += 16 / (int)sizeof(T)) {
      const uint4 raw = *(const uint4*)(km + e);
      const T* v = (const T*)&raw;
#pragma unroll
      for (int j = 0; j < 16 / (int)sizeof(T); ++j) kv[e + j] = Elem<T>::load(v + j);
    }
#pragma unroll
    for (int e = 0; e < SL / 2; ++e) {
      h2[e] = ((const double2*)hi)[e];
      l2[e] = ((const double2*)lo)[e];
    }
    double acc = 0.0;
#pragma unroll
    for (int e = 0; e < SL / 2; ++e)
      acc += (double)kv[2 * e] * (h2[e].x - l2[e].x) + (double)kv[2 * e + 1] * (h2[e].y - l2[e].y);
    acc += __shfl_xor(acc, 1);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 4);
    if (sl == 0) r[t] = (acc != acc) ? -__builtin_inf() : acc;  // NaN ranks lowest
  }
  __syncthreads();

  // Rank under the strict order (larger r first, then lower offset); the r_k
  // tokens of rank < r_k are the representatives.  One thread per token; the
  // comparisons run over pairs of LDS values, several loads in flight.
  // (one thread per token: lbs <= 256 <= NT)
  const int t = tid;
  bool sel = false;
  if (t < lbs) {
    const double rt = r[t];
    int rank = 0;
    const int pairs = lbs >> 1;
    int u2 = 0;
    for (; u2 + 4 <= pairs; u2 += 4) {
      double2 x[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) x[j] = ((const double2*)r)[u2 + j];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int u = 2 * (u2 + j);
        rank += (x[j].x > rt) || (x[j].x == rt && u < t);
        rank += (x[j].y > rt) || (x[j].y == rt && u + 1 < t);
      }
    }
    for (int u = 2 * u2; u < lbs; ++u) {
      const double ru = r[u];
      rank += (ru > rt) || (ru == rt && u < t);
    }
    sel = rank < a.n_repr;
  }
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


}  // namespace infllm
