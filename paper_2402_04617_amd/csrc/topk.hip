// Top-k unit lookup (Section 3.2: only the k_m units of highest relevance are loaded).
//
// One workgroup per row.  Scores map to order-preserving 32-bit keys; a 4-pass
// MSB-first radix select (256-bin LDS histograms) finds the k-th largest key T
// and how many keys equal to T to keep; a pass in index order then keeps every
// key > T and the lowest-indexed keys == T, writing survivors with a block-wide
// ballot scan so the output is ascending by construction.  Deterministic.
#include "launch.h"

namespace infllm {
namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / 64;

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

__global__ void __launch_bounds__(kThreads) topk_kernel(const float* __restrict__ scores, int n, int k,
                                                        int32_t* __restrict__ idx) {
  const int row = blockIdx.x;
  const float* s = scores + (int64_t)row * n;
  int32_t* out = idx + (int64_t)row * k;
  const int k_eff = min(k, n);
  for (int j = k_eff + threadIdx.x; j < k; j += kThreads) out[j] = -1;
  if (k_eff == 0) return;

  __shared__ uint32_t hist[256];
  __shared__ uint32_t sh_digit, sh_remaining;
  __shared__ int wave_tot[kWaves];

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

}  // namespace

hipError_t launch_select_topk(int rows, const float* scores, int n_units, int k, int32_t* idx,
                              hipStream_t s) {
  if (rows == 0 || k == 0) return hipSuccess;
  hipLaunchKernelGGL(topk_kernel, dim3(rows), dim3(kThreads), 0, s, scores, n_units, k, idx);
  return hipGetLastError();
}

}  // namespace infllm
