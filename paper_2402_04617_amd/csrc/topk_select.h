// Top-k unit lookup (Section 3.2: only the k_m units of highest relevance are loaded):
// the workgroup-level select, shared by the selection kernel and the attention
// kernel's prologue (which may select its kv head's units itself).
//
// One workgroup per row.  Scores map to order-preserving 32-bit keys; a 4-pass
// MSB-first radix select (256-bin LDS histograms) finds the k-th largest key T
// and how many keys equal to T to keep; a pass in index order then keeps every
// key > T and the lowest-indexed keys == T, writing survivors with a block-wide
// ballot scan so the output is ascending by construction.  Deterministic.
// Rows of up to kThreads*kMaxPer keys keep their keys in registers for all
// passes (radix_select_reg); longer rows re-read them from memory.  Rows of
// several keys per thread first narrow the keys to the candidates at or above
// the selection threshold of the per-thread maxima (filtered_select).
#pragma once
#include "launch.h"

namespace infllm {
namespace {
namespace tk {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;
constexpr int kMaxPer = 16;  // most keys per thread held in registers
constexpr int kCountMax = 128;  // most filter candidates ranked by counting

__device__ __forceinline__ uint32_t order_key(float x) {
  if (x != x) return 0u;        // NaN below everything
  if (x == 0.0f) x = 0.0f;      // -0 == +0
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive block scan of a predicate in thread order; returns this thread's
// exclusive prefix and sets *total.  Uses (and ends with) a barrier.
__device__ __forceinline__ int block_scan(bool pred, int* wave_tot, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long m = __ballot(pred);
  const int pre = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wave_tot[wave] = __popcll(m);
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int c = wave_tot[w];
    off += (w < wave) ? c : 0;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  return off + pre;
}

// Radix-select path (see above); s, out: this row.  (Unused by the attention
// kernels that include this header.)
[[maybe_unused]] __device__ void radix_select(const float* __restrict__ s, int n, int k_eff, int32_t* __restrict__ out,
                             int* wave_tot) {
  __shared__ uint32_t hist[256];
  __shared__ uint32_t sh_digit, sh_remaining;

  const bool all = (k_eff == n);
  uint32_t thr = 0;
  int need_eq = 0;
  if (!all) {
    uint32_t prefix = 0, mask = 0;
    int remaining = k_eff;
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int j = threadIdx.x; j < 256; j += kThreads) hist[j] = 0;
      __syncthreads();
      for (int i = threadIdx.x; i < n; i += kThreads) {
        const uint32_t key = order_key(s[i]);
        if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (threadIdx.x < 64) {
        // lane l owns bins 4l..4l+3; suffix sums give counts of keys >= each bin
        const int l = threadIdx.x;
        const uint32_t h0 = hist[4 * l], h1 = hist[4 * l + 1], h2 = hist[4 * l + 2], h3 = hist[4 * l + 3];
        uint32_t own = h0 + h1 + h2 + h3;
        uint32_t suf = own;  // inclusive suffix over lanes >= l
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const uint32_t x = __shfl_down(suf, o);
          suf += (l + o < 64) ? x : 0u;
        }
        const uint32_t above = suf - own;  // keys in bins > 4l+3
        const uint32_t ge3 = above + h3, ge2 = ge3 + h2, ge1 = ge2 + h1, ge0 = ge1 + h0;
        const uint32_t rem = (uint32_t)remaining;
        // the digit d* with count(>= d*) >= rem > count(> d*)
        if (ge3 >= rem && above < rem) { sh_digit = 4 * l + 3; sh_remaining = rem - above; }
        if (ge2 >= rem && ge3 < rem) { sh_digit = 4 * l + 2; sh_remaining = rem - ge3; }
        if (ge1 >= rem && ge2 < rem) { sh_digit = 4 * l + 1; sh_remaining = rem - ge2; }
        if (ge0 >= rem && ge1 < rem) { sh_digit = 4 * l; sh_remaining = rem - ge1; }
      }
      __syncthreads();
      prefix |= sh_digit << shift;
      mask |= 255u << shift;
      remaining = (int)sh_remaining;
      __syncthreads();
    }
    thr = prefix;
    need_eq = remaining;
  }

  int base_eq = 0, base_sel = 0;
  for (int tile = 0; tile < n; tile += kThreads) {
    const int i = tile + threadIdx.x;
    const bool valid = i < n;
    const uint32_t key = valid ? order_key(s[i]) : 0u;
    const bool is_eq = valid && !all && key == thr;
    int tot_eq;
    const int eq_rank = base_eq + block_scan(is_eq, wave_tot, &tot_eq);
    const bool keep = valid && (all || key > thr || (is_eq && eq_rank < need_eq));
    int tot_sel;
    const int pos = base_sel + block_scan(keep, wave_tot, &tot_sel);
    if (keep && pos < k_eff) out[pos] = i;
    base_eq += tot_eq;
    base_sel += tot_sel;
  }
}

// Exclusive ranks, in index order, of the set predicates of PER strided tiles
// (thread t holds element t + j*kThreads of tile j): per-(tile, wave) ballot
// counts through LDS, two barriers in all.
template <int PER>
__device__ __forceinline__ void tiled_scan(const bool (&pred)[PER], int (&rank)[PER], int* total) {
  __shared__ int cnt[PER][kWaves];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long below = (1ull << lane) - 1ull;
  unsigned long long m[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    m[j] = __ballot(pred[j]);
    if (lane == 0) cnt[j][wave] = __popcll(m[j]);
  }
  __syncthreads();
  int base = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    int before = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const int c = cnt[j][w];
      before += (w < wave) ? c : 0;
      tot += c;
    }
    rank[j] = base + before + __popcll(m[j] & below);
    base += tot;
  }
  *total = base;
  __syncthreads();  // cnt may be written again by the next scan
}

// Threshold of the radix select over keys held PER per thread (thread t: keys
// t, t + kThreads, ...; live[j] marks the ones taking part): the histogram of a
// pass is built with one atomic per wave where the wave's live digits agree
// (typical of the leading digits), histograms are double-buffered (two barriers
// per pass), and the passes stop early once every key sharing the resolved
// prefix is kept.  On return thr is the k_eff-th largest live key and
// `remaining` the number of live keys equal to it to keep (lowest indices
// first) -- or, with ge_all set, thr is that prefix with its low bits zero and
// exactly k_eff live keys are >= thr.  Either way at least k_eff live keys are
// >= thr.  With MAXP < 4 the passes stop after MAXP digits: thr is then only
// such a lower bound (the resolved prefix, low bits zero; ge_all is false).
// Requires 0 < k_eff <= the live count.
template <int PER, int MAXP = 4, typename Live>
__device__ void radix_threshold(const uint32_t (&key)[PER], Live live_in, int k_eff, uint32_t& thr,
                                int& remaining_out, bool& ge_all) {
  __shared__ uint32_t hist[2][256];
  __shared__ uint32_t sh_digit, sh_remaining, sh_eq_total;
  const int t = threadIdx.x, lane = t & 63;
  for (int j = t; j < 256; j += kThreads) hist[0][j] = 0;
  __syncthreads();
  uint32_t prefix = 0, mask = 0;
  int remaining = k_eff;
  uint32_t eq_total = 0;
  for (int pass = 0; pass < MAXP; ++pass) {
    const int shift = 24 - 8 * pass;
    uint32_t* h = hist[pass & 1];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const bool live = live_in(j) && (key[j] & mask) == prefix;
      const uint32_t d = (key[j] >> shift) & 255u;
      const unsigned long long lm = __ballot(live);
      if (lm == 0) continue;
      const uint32_t d0 = (uint32_t)__builtin_amdgcn_readlane((int)d, __builtin_ctzll(lm));
      if (__ballot(live && d != d0) == 0) {
        if (lane == 0) atomicAdd(&h[d0], (uint32_t)__popcll(lm));
      } else if (live) {
        atomicAdd(&h[d], 1u);
      }
    }
    __syncthreads();
    if (t < 64) {
      // lane l owns bins 4l..4l+3; suffix sums give counts of keys >= each bin
      const uint32_t h0 = h[4 * t], h1 = h[4 * t + 1], h2 = h[4 * t + 2], h3 = h[4 * t + 3];
      const uint32_t own = h0 + h1 + h2 + h3;
      uint32_t suf = own;  // inclusive suffix over lanes >= l
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t x = __shfl_down(suf, o);
        suf += (t + o < 64) ? x : 0u;
      }
      const uint32_t above = suf - own;  // keys in bins > 4l+3
      const uint32_t ge3 = above + h3, ge2 = ge3 + h2, ge1 = ge2 + h1, ge0 = ge1 + h0;
      const uint32_t rem = (uint32_t)remaining;
      // the digit d* with count(>= d*) >= rem > count(> d*)
      if (ge3 >= rem && above < rem) { sh_digit = 4 * t + 3; sh_remaining = rem - above; sh_eq_total = h3; }
      if (ge2 >= rem && ge3 < rem) { sh_digit = 4 * t + 2; sh_remaining = rem - ge3; sh_eq_total = h2; }
      if (ge1 >= rem && ge2 < rem) { sh_digit = 4 * t + 1; sh_remaining = rem - ge2; sh_eq_total = h1; }
      if (ge0 >= rem && ge1 < rem) { sh_digit = 4 * t; sh_remaining = rem - ge1; sh_eq_total = h0; }
    } else {
      for (int j = t - 64; j < 256; j += kThreads - 64) hist[(pass + 1) & 1][j] = 0;
    }
    __syncthreads();
    prefix |= sh_digit << shift;
    mask |= 255u << shift;
    remaining = (int)sh_remaining;
    eq_total = sh_eq_total;
    // Every key with this prefix is kept: the prefix (low bits zero) is already a
    // threshold that keeps exactly k_eff keys, so the remaining passes are skipped.
    if ((uint32_t)remaining == eq_total) break;
  }
  // the shared words are read again by the next call
  __syncthreads();
  thr = prefix;
  remaining_out = remaining;
  ge_all = (uint32_t)remaining == eq_total;
}

// The selection given a threshold: keep the live keys above thr and the first
// `remaining` equal to it in element order (element j of thread t is the
// (j * kThreads + t)-th; ranks from per-(tile, wave) ballot counts), and write
// the pos-th kept element's index ix(j) to out[pos] -- ascending when ix is.
template <int PER, typename Live, typename Index>
__device__ void write_selection(const uint32_t (&key)[PER], Live live, Index ix, uint32_t thr, int remaining,
                                bool ge_all, int k_eff, int32_t* __restrict__ out) {
  bool keep[PER];
  if (ge_all) {
#pragma unroll
    for (int j = 0; j < PER; ++j) keep[j] = live(j) && key[j] >= thr;
  } else {
    bool eq[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) eq[j] = live(j) && key[j] == thr;
    int eq_rank[PER], tot;
    tiled_scan<PER>(eq, eq_rank, &tot);
#pragma unroll
    for (int j = 0; j < PER; ++j) keep[j] = live(j) && (key[j] > thr || (eq[j] && eq_rank[j] < remaining));
  }
  int pos[PER], tot;
  tiled_scan<PER>(keep, pos, &tot);
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (keep[j] && pos[j] < k_eff) out[pos[j]] = ix(j);
}

// Long rows (several keys per thread, k_eff <= kThreads): a cheap filter first.
// Let m be a key with at least k_eff per-thread maxima >= m (the 16-bit prefix
// two radix passes over the maxima resolve): those k_eff maxima are distinct
// keys >= m, so the row's k_eff-th largest key T is >= m, and every key the
// selection keeps (the keys > T and the lowest-indexed keys == T) is among the
// candidates >= m.  The candidates are compacted in index order and the
// selection is run on them, one per thread: few candidates rank themselves by
// counting (rank = candidates with a larger key, or an equal key at a lower
// index; kept iff rank < k_eff), more run the radix select.  Either way the
// result is the one the full select gives.  Returns false (workgroup-uniform)
// when more than kThreads candidates remain, e.g. on massive ties; the caller
// then selects over all keys.
template <int PER>
__device__ bool filtered_select(const uint32_t (&key)[PER], int n, int k_eff, int32_t* __restrict__ out) {
  __shared__ uint32_t ckey[kThreads];
  __shared__ int32_t cidx[kThreads];
  const int t = threadIdx.x;
  auto valid = [&](int j) { return t + j * kThreads < n; };
  uint32_t mx[1] = {0u};
#pragma unroll
  for (int j = 0; j < PER; ++j)
    if (valid(j)) mx[0] = max(mx[0], key[j]);
  uint32_t m;
  int rem;
  bool ge;
  radix_threshold<1, 2>(mx, [&](int) { return t < n; }, k_eff, m, rem, ge);  // thread t holds key t
  // Compaction in element order: per-(tile, wave) candidate counts, their
  // exclusive prefix in element order (tile-major), then each candidate's slot
  // from its wave's ballot.  The predicate is recomputed rather than kept.
  __shared__ int cbase[PER * kWaves + 1];
  const int lane = t & 63, wave = t >> 6;
  auto cand = [&](int j) { return valid(j) && key[j] >= m; };
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const unsigned long long b = __ballot(cand(j));
    if (lane == 0) cbase[j * kWaves + wave] = __popcll(b);
  }
  __syncthreads();
  if (t < 64) {
    // lane l takes entries 2l and 2l+1 (PER * kWaves <= 128)
    constexpr int NE = PER * kWaves;
    const int c0 = 2 * t < NE ? cbase[2 * t] : 0, c1 = 2 * t + 1 < NE ? cbase[2 * t + 1] : 0;
    int inc = c0 + c1;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int x = __shfl_up(inc, o);
      inc += t >= o ? x : 0;
    }
    if (2 * t < NE) cbase[2 * t] = inc - c0 - c1;
    if (2 * t + 1 < NE) cbase[2 * t + 1] = inc - c1;
    if (t == 63) cbase[NE] = inc;
  }
  __syncthreads();
  const int n_cand = cbase[PER * kWaves];
  if (n_cand > kThreads) return false;
  const unsigned long long below = (1ull << lane) - 1ull;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const bool c = cand(j);
    const unsigned long long b = __ballot(c);
    if (c) {
      const int r = cbase[j * kWaves + wave] + __popcll(b & below);
      ckey[r] = key[j];
      cidx[r] = t + j * kThreads;
    }
  }
  __syncthreads();
  const bool live = t < n_cand;
  const uint32_t ck[1] = {live ? ckey[t] : 0u};
  const int ci = live ? cidx[t] : 0;
  if (n_cand <= kCountMax) {
    int rank = 0;
    for (int c = 0; c < n_cand; ++c) {
      const uint32_t kc = ckey[c];  // same address across the wave: one broadcast read
      rank += (kc > ck[0] || (kc == ck[0] && c < t)) ? 1 : 0;
    }
    __shared__ int wave_tot[kWaves];
    int tot;
    const bool keep = live && rank < k_eff;
    const int pos = block_scan(keep, wave_tot, &tot);
    if (keep) out[pos] = ci;
    return true;
  }
  uint32_t thr;
  radix_threshold<1>(ck, [&](int) { return live; }, k_eff, thr, rem, ge);
  write_selection<1>(ck, [&](int) { return live; }, [&](int) { return ci; }, thr, rem, ge, k_eff, out);
  return true;
}

// Common path: the radix select with the row's keys held in registers (thread
// t: keys t, t + kThreads, ...; read once); rows of 4+ keys per thread try the
// filter above first.
template <int PER>
__device__ void radix_select_reg(const float* __restrict__ s, int n, int k_eff, int32_t* __restrict__ out) {
  const int t = threadIdx.x;
  uint32_t key[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) key[j] = order_key(s[min(t + j * kThreads, n - 1)]);
  if constexpr (PER >= 4) {
    if (k_eff <= kThreads && filtered_select<PER>(key, n, k_eff, out)) return;
  }
  auto valid = [&](int j) { return t + j * kThreads < n; };
  uint32_t thr;
  int rem;
  bool ge;
  radix_threshold<PER>(key, valid, k_eff, thr, rem, ge);
  write_selection<PER>(key, valid, [&](int j) { return t + j * kThreads; }, thr, rem, ge, k_eff, out);
}

}  // namespace tk
}  // namespace
}  // namespace infllm
