// Append of the current tokens, in one launch:
//  - K/V rows of the chunk into the token-ordered store (copy blocks);
//  - the running group-query sum into the float64 ring that unit construction
//    reads (scan blocks), and optionally the chunk's group-query total Qbar,
//    which is exactly what unit scoring needs (the scan total, for free).
//
// The representative score of Section 3.2 needs, for every token t, the window
// sum W_t = sum_{j=1..l_L} sum_{h in group} q^h_{t+j}.  With the running sum
// Pi_p = sum_{p'<=p} sum_h q^h_{p'} kept per position, W_t is one difference of
// two ring slots, so its cost does not grow with l_L; float64 keeps the
// difference of two large running sums exact to ~1e-16.  The scan forms it as
// soon as position p = t + l_L arrives and stores k_t . W_t per 8-dim slice
// (rpart), which is all that unit construction reads later.
//
// In the whole-step path the same launch also carries the unit-construction
// blocks of the units evicted since the previous step (see unit_build.h): they
// read ring slots of earlier positions, which the chunk's new slots cannot
// overwrite when the ring is large enough (checked on the host), so the two
// latency-bound jobs overlap instead of running back to back.
//
// Scan block: one (sequence*kv head, 8-dim slice); 512 threads = 256 position
// segments x 2 halves of 4 dims.  Each thread first issues every load of its
// segment (kSeg positions: the group's query pieces, and in the streaming case
// the running sums and keys of the tokens t = p - l_L), then sums in float64; a
// DPP scan over each 32-lane half of a wave and an LDS pass over the 8 waves give
// the segment offsets, and each thread writes its kSeg ring rows.  (Per thread the
// float64 work is a long dependent chain; 4 dims per thread keeps it short enough
// that the scan ends with the copy and unit-construction blocks.)  Chunks of a few
// positions (decoding) use thin scan blocks instead, one thread per
// (sequence*kv head, dim).  Copy blocks load all their vectors before storing any.
#include <cstring>

#include "qsum.h"
#include "unit_build.h"

namespace infllm {
namespace {

constexpr int kThreads = 512;                  // threads of every block of the launch (two waves per SIMD;
                                               // a scan thread keeps a whole segment's loads in flight)
constexpr int kWaves = kThreads / 64;
constexpr int kSeg = 2;                        // positions per thread per tile: a 512-position chunk is one tile
constexpr int kTile = (kThreads / 2) * kSeg;   // positions per scan tile
constexpr int kCopyPerThread = 4;              // 16-byte vectors per thread in copy blocks
constexpr int kThinMaxQ = 8;                   // chunks this short take the one-thread-per-dim scan
constexpr int kDPT = kRpartDims / 2;           // dimensions per scan thread (a slice's two halves)

// R(pos) applied to one 16-byte vector of consecutive dimensions starting at the
// even dimension 2*pair0 (positional remap): 4 bf16 pairs or 2 float32 pairs.
template <typename T>
__device__ __forceinline__ uint4 rotate_vec(const uint4 w, int64_t pos, int pair0, const RopeArgs& r) {
  uint32_t in[4] = {w.x, w.y, w.z, w.w}, out[4];
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float c, sn;
      rope_cos_sin(r, pos, pair0 + j, c, sn);
      const float x0 = __uint_as_float(in[j] << 16), x1 = __uint_as_float(in[j] & 0xFFFF0000u);
      out[j] = (uint32_t)f32_to_bf16(x0 * c - x1 * sn) | ((uint32_t)f32_to_bf16(x0 * sn + x1 * c) << 16);
    }
  } else {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float c, sn;
      rope_cos_sin(r, pos, pair0 + j, c, sn);
      const float x0 = __uint_as_float(in[2 * j]), x1 = __uint_as_float(in[2 * j + 1]);
      out[2 * j] = __float_as_uint(x0 * c - x1 * sn);
      out[2 * j + 1] = __float_as_uint(x0 * sn + x1 * c);
    }
  }
  return make_uint4(out[0], out[1], out[2], out[3]);
}

// kDPT consecutive elements of a query or key row as raw words (kDPT*sizeof(T)
// bytes: one 8-byte load for bf16, one 16-byte load for float32).
template <typename T>
struct RawD {
  uint32_t w[kDPT * sizeof(T) / 4];
};
template <typename T>
__device__ __forceinline__ RawD<T> load_rawd(const T* p) {
  RawD<T> r;
  if constexpr (kDPT * sizeof(T) == 8) {
    const uint2 v = *(const uint2*)p;
    r.w[0] = v.x;
    r.w[1] = v.y;
  } else {
    static_assert(kDPT * sizeof(T) == 16, "one 8- or 16-byte piece per thread");
    const uint4 v = *(const uint4*)p;
    r.w[0] = v.x;
    r.w[1] = v.y;
    r.w[2] = v.z;
    r.w[3] = v.w;
  }
  return r;
}
template <typename T>
__device__ __forceinline__ void rawd_to_float(const RawD<T>& r, float* out) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int e = 0; e < kDPT / 2; ++e) {
      out[2 * e] = __uint_as_float(r.w[e] << 16);
      out[2 * e + 1] = __uint_as_float(r.w[e] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int e = 0; e < kDPT; ++e) out[e] = __uint_as_float(r.w[e]);
  }
}
// R(pos) on kDPT consecutive dimensions (kDPT/2 pairs from pair0), float64 or float.
template <typename V>
__device__ __forceinline__ void rotate_d(V (&x)[kDPT], int64_t pos, int pair0, const RopeArgs& r) {
#pragma unroll
  for (int j = 0; j < kDPT / 2; ++j) {
    float c, sn;
    rope_cos_sin(r, pos, pair0 + j, c, sn);
    const V x0 = x[2 * j], x1 = x[2 * j + 1];
    x[2 * j] = x0 * (V)c - x1 * (V)sn;
    x[2 * j + 1] = x0 * (V)sn + x1 * (V)c;
  }
}

// Cross-lane moves of a float64 for the scan: DPP (two 32-bit halves) on the
// vector ALU instead of LDS permutes.  Lanes whose source lies outside the
// pattern read 0.  CTRL: row_shr:n = 0x110 + n; row_bcast:15 = 0x142.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_f64(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, ROW_MASK, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, ROW_MASK, 0xF, false);
  return __longlong_as_double((long long)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}
// Inclusive sum over lanes [32h, lane] of each 32-lane half h.
__device__ __forceinline__ double half_wave_scan(double x) {
  x += dpp_f64<0x111, 0xF>(x);
  x += dpp_f64<0x112, 0xF>(x);
  x += dpp_f64<0x114, 0xF>(x);
  x += dpp_f64<0x118, 0xF>(x);
  x += dpp_f64<0x142, 0xA>(x);  // rows 1 and 3 add the last lane of rows 0 and 2
  return x;
}
// x of lane l plus x of lane l ^ 32, the same sum in both lanes.
__device__ __forceinline__ double add_halves(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const auto lo = __builtin_amdgcn_permlane32_swap((uint32_t)u, (uint32_t)u, false, false);
  const auto hi = __builtin_amdgcn_permlane32_swap((uint32_t)(u >> 32), (uint32_t)(u >> 32), false, false);
  const double a = __longlong_as_double((long long)(((uint64_t)hi[0] << 32) | lo[0]));
  const double b = __longlong_as_double((long long)(((uint64_t)hi[1] << 32) | lo[1]));
  return a + b;
}

// Block roles along the 1-D grid: [unit construction | query sum | scan | copy].
struct AppendGrid {
  int n_build;          // unit-construction blocks (n_new * batch * Hkv), 0 when not fused
  int n_qsum;           // query-sum blocks (Mean Repr: parts * batch * Hkv), 0 otherwise
  int qsum_parts;
  int n_scan;           // scan blocks
  bool thin;            // scan blocks are thin (one thread per (sequence*kv head, dim))
  int n_copy_per_head;  // copy blocks per (sequence, kv head)
};

// GT: the query group size G when known at compile time (0: read it at run time).
// ROPE: the positional remap is on (a.rope.on), fixed at compile time so that
// the plain path carries none of its code.
template <typename T, int GT, int DT, bool ROPE>
__global__ void __launch_bounds__(kThreads) append_kernel(AppendArgs a, BuildArgs ba, AppendGrid grid,
                                                          float* __restrict__ qbar) {
  const int D = a.head_dim;
  __shared__ BuildSmem bsm;
  int blk = blockIdx.x;
  if (blk < grid.n_build) {
    // ---- unit-construction role
    const int bh = ba.batch * ba.n_kv_heads;
    construct_unit<T, DT, kThreads>(ba, blk / bh, blk % bh, bsm);
    return;
  }
  blk -= grid.n_build;
  if (blk < grid.n_qsum) {
    // ---- query-sum role (Mean Repr, which has no scan): the chunk's group-query
    // partial sums that unit scoring consumes
    __shared__ QsumSmem<T, kThreads> qsm;
    qsum_block<T, kThreads>((const T*)a.q, a.q_head_stride, a.n_q_heads, a.n_kv_heads, D, a.n_q, blk % grid.qsum_parts,
                  grid.qsum_parts, blk / grid.qsum_parts, qbar, qsm);
    return;
  }
  blk -= grid.n_qsum;
  if (blk >= grid.n_scan) {
    // ---- copy role: K and V rows of the chunk into the store; each thread
    // moves kCopyPerThread 16-byte vectors of one (sequence, kv head).
    blk -= grid.n_scan;
    constexpr int VEC = 16 / sizeof(T);
    const int vec_per_head = a.n_q * D / VEC;
    const int64_t head = blk / grid.n_copy_per_head;
    const int cblk = blk % grid.n_copy_per_head;
    const int64_t past = seq_past(a, (int)(head / a.n_kv_heads));
    const uint4* src_k = (const uint4*)a.k_src + head * (a.kv_head_stride / VEC);
    const uint4* src_v = (const uint4*)a.v_src + head * (a.kv_head_stride / VEC);
    uint4* dst_k = (uint4*)a.k_store + head * (a.capacity * D / VEC) + past * D / VEC;
    uint4* dst_v = (uint4*)a.v_store + head * (a.capacity * D / VEC) + past * D / VEC;
    const int base = cblk * kThreads * kCopyPerThread + threadIdx.x;
    // all loads first (clamped indices), then the guarded stores
    const int e0 = base, e1 = base + kThreads, e2 = base + 2 * kThreads, e3 = base + 3 * kThreads;
    static_assert(kCopyPerThread == 4, "copy role moves four vectors per thread");
    const int last = vec_per_head - 1;
    const uint4 k0 = src_k[min(e0, last)], k1 = src_k[min(e1, last)], k2 = src_k[min(e2, last)],
                k3 = src_k[min(e3, last)];
    const uint4 v0 = src_v[min(e0, last)], v1 = src_v[min(e1, last)], v2 = src_v[min(e2, last)],
                v3 = src_v[min(e3, last)];
    if (e0 < vec_per_head) { dst_k[e0] = k0; dst_v[e0] = v0; }
    if (e1 < vec_per_head) { dst_k[e1] = k1; dst_v[e1] = v1; }
    if (e2 < vec_per_head) { dst_k[e2] = k2; dst_v[e2] = v2; }
    if (e3 < vec_per_head) { dst_k[e3] = k3; dst_v[e3] = v3; }
    if (ROPE) {
      // positional remap: the keys rotated to their own positions go to k_rot
      uint4* dst_r = (uint4*)a.k_rot + head * (a.capacity * D / VEC) + past * D / VEC;
      const int vpp = D / VEC;  // vectors per position
      auto rot = [&](int e, const uint4& w) {
        if (e < vec_per_head)
          dst_r[e] = rotate_vec<T>(w, past + e / vpp, (e % vpp) * (VEC / 2), a.rope);
      };
      rot(e0, k0);
      rot(e1, k1);
      rot(e2, k2);
      rot(e3, k3);
    }
    return;
  }

  if (grid.thin) {
    // ---- thin scan role, for chunks of at most kThinMaxQ positions (decoding):
    // one thread per (sequence*kv head, dim) walks the positions in order.  The
    // 16 threads of a slice are adjacent lanes, so the partial score of a slice
    // is a 16-lane sum.
    const int gid = blk * kThreads + threadIdx.x;
    if (gid >= a.batch * a.n_kv_heads * D) return;  // whole waves: the total is a multiple of 64
    const int bg = gid / D, d = gid - bg * D;
    const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
    const int64_t past = seq_past(a, b);
    const int G = GT > 0 ? GT : a.n_q_heads / a.n_kv_heads;
    const T* qb = (const T*)a.q + (int64_t)(b * a.n_q_heads + g * G) * a.q_head_stride + d;
    double* col = a.qprefix + (int64_t)bg * a.ring * D + d;
    const int slot0 = (int)(past % a.ring);
    // every load that does not depend on this launch's writes is issued first
    const T* kread = (const T*)a.k_store;
    double x[kThinMaxQ], ht[kThinMaxQ];
    float kt[kThinMaxQ];
#pragma unroll
    for (int i = 0; i < kThinMaxQ; ++i) {
      x[i] = 0.0;
      ht[i] = 0.0;
      kt[i] = 0.f;
      if (i < a.n_q) {
        for (int h = 0; h < G; ++h) x[i] += (double)Elem<T>::load(qb + h * a.q_head_stride + (int64_t)i * D);
        const int64_t t = past + i - a.n_local;
        if (t >= a.n_init && t < past) {
          const int sp = slot0 + i - (slot0 + i >= a.ring ? a.ring : 0);
          const int st = sp - a.n_local + (sp < a.n_local ? a.ring : 0);  // n_local < ring
          ht[i] = col[(int64_t)st * D];
          kt[i] = Elem<T>::load(kread + ((int64_t)bg * a.capacity + t) * D + d);
        }
      }
    }
    double run = 0.0;
    if (past > 0) run = col[(int64_t)(slot0 == 0 ? a.ring - 1 : slot0 - 1) * D];
    const double base = run;
    float raw_tot = 0.f;  // the chunk's unrotated query sum (remap: the ring holds rotated sums)
    // R(pos) on dimension d of a pair split over lanes d, d^1 (uniform branch: pos is per position)
    auto rot_lane = [&](double v, int64_t pos) -> double {
      const double w = __shfl_xor(v, 1);
      float c, sn;
      rope_cos_sin(a.rope, pos, d >> 1, c, sn);
      return (d & 1) ? w * (double)sn + v * (double)c : v * (double)c - w * (double)sn;
    };
#pragma unroll
    for (int i = 0; i < kThinMaxQ; ++i) {
      if (i >= a.n_q) continue;  // (not break: the loop stays unrolled, the arrays in registers)
      raw_tot += (float)x[i];
      if (ROPE) x[i] = rot_lane(x[i], past + i);
      run += x[i];
      const int sp = slot0 + i - (slot0 + i >= a.ring ? a.ring : 0);
      col[(int64_t)sp * D] = run;
      const int64_t t = past + i - a.n_local;
      if (t >= a.n_init) {
        double h = ht[i], k = kt[i];
        if (t >= past) {
          // token of this chunk: its running sum was written by this thread above
          const int st = sp - a.n_local + (sp < a.n_local ? a.ring : 0);
          h = col[(int64_t)st * D];
          k = Elem<T>::load((const T*)a.k_src + (int64_t)bg * a.kv_head_stride + (t - past) * D + d);
        }
        // positional remap: the input key turned to its own position, unrounded
        if (ROPE) k = rot_lane(k, t);
        double part = k * (run - h);
#pragma unroll
        for (int o = 1; o < kRpartDims; o <<= 1) part += __shfl_xor(part, o);
        if ((d % kRpartDims) == 0)
          a.rpart[((int64_t)bg * (D / kRpartDims) + d / kRpartDims) * a.ring + (int)(t % a.ring)] = part;
      }
    }
    if (qbar != nullptr) qbar[(int64_t)bg * D + d] = ROPE ? raw_tot : (float)(run - base);
    return;
  }

  // ---- scan role.  The slice blocks of one (sequence, kv head) read pieces of
  // the same 256-byte query and key rows: they are placed on one XCD (blocks whose
  // ids agree modulo the XCD count share one), so that its L2 fetches each row from
  // HBM once instead of once per slice.
  const int slices = D / kRpartDims;
  if (grid.n_scan % kNumXcd == 0) blk = xcd_logical_block(blk, grid.n_scan);
  const int bg = blk / slices;
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
  const int64_t past = seq_past(a, b);
  // lanes [0, 32) of a wave take the slice's first kDPT dims, lanes [32, 64) the
  // other kDPT, for the same 32 position segments (a segment scan is a 32-lane scan)
  const int half = (threadIdx.x >> 5) & 1, seg = (threadIdx.x >> 6) * 32 + (threadIdx.x & 31);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int slice = blk - bg * slices;
  const int d0 = slice * kRpartDims + half * kDPT;
  const int G = GT > 0 ? GT : a.n_q_heads / a.n_kv_heads;
  const T* qb = (const T*)a.q + (int64_t)(b * a.n_q_heads + g * G) * a.q_head_stride + d0;
  double* ring = a.qprefix + (int64_t)bg * a.ring * D + d0;

  __shared__ double wave_tot[kWaves][2][kDPT];
  __shared__ float wave_raw[kWaves][2][kDPT];
  // stored keys as given (unrotated); under the remap each is turned to its own
  // position here in float32, never through the bf16-rounded k_rot copy
  const T* kread = (const T*)a.k_store;
  float raw_acc[kDPT];  // unrotated query sum of this thread's positions (the chunk total feeds scoring)
#pragma unroll
  for (int e = 0; e < kDPT; ++e) raw_acc[e] = 0.f;
  const int slot0 = (int)(past % a.ring);  // ring > n_q: slot0 + i wraps at most once
  double base[kDPT], carry[kDPT];
  if (past > 0) {
    const double* src = ring + (int64_t)(slot0 == 0 ? a.ring - 1 : slot0 - 1) * D;
#pragma unroll
    for (int e = 0; e < kDPT; ++e) base[e] = src[e];
  } else {
#pragma unroll
    for (int e = 0; e < kDPT; ++e) base[e] = 0.0;
  }
#pragma unroll
  for (int e = 0; e < kDPT; ++e) carry[e] = base[e];
  // (no barrier: the slots this launch writes, positions past .. past + n_q - 1, never
  // alias slot past - 1 or the slots of the tokens t = p - l_L it reads, since the host
  // checked ring >= l_L + n_q; so the base loads stay in flight with the tile's loads)

  constexpr int GQ = GT > 0 ? GT : 1;  // query pieces loaded up front per position
  constexpr int NP = kDPT / 2;          // dimension pairs (double2) per thread
  for (int t0 = 0; t0 < a.n_q; t0 += kTile) {
    const int i0 = t0 + seg * kSeg;
    // When every token t = p - l_L of this tile precedes the chunk (l_L >= the
    // tile's end, the streaming case), its running sum and key are loaded now,
    // together with the queries, and its partial score is formed right where
    // the new running sum is written.  Loads use clamped indices (the values of
    // inactive positions are never used).
    const bool early = t0 + kTile <= a.n_local;
    RawD<T> qr[kSeg][GQ];
    double2 ht[kSeg][NP];
    RawD<T> kr[kSeg];
    int slot_t[kSeg];  // ring slot of token t = p - l_L
#pragma unroll
    for (int s = 0; s < kSeg; ++s) {
      const int ic = min(i0 + s, a.n_q - 1);
#pragma unroll
      for (int h = 0; h < GQ; ++h) qr[s][h] = load_rawd<T>(qb + h * a.q_head_stride + (int64_t)ic * D);
    }
    if (early) {
#pragma unroll
      for (int s = 0; s < kSeg; ++s) {
        const int ic = min(i0 + s, a.n_q - 1);
        const int sp = slot0 + ic - (slot0 + ic >= a.ring ? a.ring : 0);
        const int st = sp - a.n_local + (sp < a.n_local ? a.ring : 0);  // n_local < ring
        slot_t[s] = st;
        const double2* src = (const double2*)(ring + (int64_t)st * D);
#pragma unroll
        for (int e = 0; e < NP; ++e) ht[s][e] = src[e];
        int64_t tk = past + ic - a.n_local;
        tk = tk < 0 ? 0 : tk;
        kr[s] = load_rawd<T>(kread + ((int64_t)bg * a.capacity + tk) * D + d0);
      }
    }
    double run[kSeg][kDPT];
    double tot[kDPT];
#pragma unroll
    for (int e = 0; e < kDPT; ++e) tot[e] = 0.0;
#pragma unroll
    for (int s = 0; s < kSeg; ++s) {
      const int i = min(i0 + s, a.n_q - 1);
      const bool valid = i0 + s < a.n_q;
      double x[kDPT];
#pragma unroll
      for (int e = 0; e < kDPT; ++e) x[e] = 0.0;
      if constexpr (GT > 0) {
#pragma unroll
        for (int h = 0; h < GT; ++h) {
          float y[kDPT];
          rawd_to_float<T>(qr[s][h], y);
#pragma unroll
          for (int e = 0; e < kDPT; ++e) x[e] += (double)y[e];
        }
      } else {
        for (int h = 0; h < G; ++h) {
          float y[kDPT];
          rawd_to_float<T>(h == 0 ? qr[s][0] : load_rawd<T>(qb + h * a.q_head_stride + (int64_t)i * D), y);
#pragma unroll
          for (int e = 0; e < kDPT; ++e) x[e] += (double)y[e];
        }
      }
      if (ROPE) {
        // the ring sums the queries rotated to their positions; scoring takes the plain sum
#pragma unroll
        for (int e = 0; e < kDPT; ++e) raw_acc[e] += valid ? (float)x[e] : 0.f;
        rotate_d(x, past + i, d0 / 2, a.rope);
      }
#pragma unroll
      for (int e = 0; e < kDPT; ++e) {
        tot[e] += valid ? x[e] : 0.0;
        run[s][e] = tot[e];
      }
    }
    // inclusive scan of segment totals across the 32 segments of this half in the wave
    double incl[kDPT];
#pragma unroll
    for (int e = 0; e < kDPT; ++e) incl[e] = half_wave_scan(tot[e]);
    if ((lane & 31) == 31) {
#pragma unroll
      for (int e = 0; e < kDPT; ++e) wave_tot[wave][half][e] = incl[e];
    }
    __syncthreads();
    double off[kDPT], tile_tot[kDPT];
#pragma unroll
    for (int e = 0; e < kDPT; ++e) {
      off[e] = incl[e] - tot[e];
      tile_tot[e] = 0.0;
    }
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
#pragma unroll
      for (int e = 0; e < kDPT; ++e) {
        const double y = wave_tot[w][half][e];
        off[e] += (w < wave) ? y : 0.0;
        tile_tot[e] += y;
      }
    }
    double part[kSeg];
#pragma unroll
    for (int s = 0; s < kSeg; ++s) {
      const int i = i0 + s;
      float kt[kDPT];
      rawd_to_float<T>(kr[s], kt);
      if (ROPE && early) rotate_d(kt, past + i - a.n_local, d0 / 2, a.rope);
      part[s] = 0.0;
      if (i < a.n_q) {
        const int slot = slot0 + i - (slot0 + i >= a.ring ? a.ring : 0);
        double2* d2 = (double2*)(ring + (int64_t)slot * D);
#pragma unroll
        for (int e = 0; e < NP; ++e) {
          const double2 nv = make_double2(carry[2 * e] + off[2 * e] + run[s][2 * e],
                                          carry[2 * e + 1] + off[2 * e + 1] + run[s][2 * e + 1]);
          d2[e] = nv;
          if (early)
            part[s] += (double)kt[2 * e] * (nv.x - ht[s][e].x) + (double)kt[2 * e + 1] * (nv.y - ht[s][e].y);
        }
      }
    }
    if (early) {
#pragma unroll
      for (int s = 0; s < kSeg; ++s) {
        const int i = i0 + s;
        const int64_t t = past + i - a.n_local;
        part[s] = add_halves(part[s]);  // the two halves of the slice
        if (i < a.n_q && t >= a.n_init && half == 0)
          a.rpart[((int64_t)bg * slices + slice) * a.ring + slot_t[s]] = part[s];
      }
    }
#pragma unroll
    for (int e = 0; e < kDPT; ++e) carry[e] += tile_tot[e];
    __syncthreads();

    // Otherwise the partial representative scores of the tokens t = p - l_L
    // (t >= l_I) of this tile's positions p are formed now: both running sums are
    // in the ring (the barrier above published this tile's slots; the host
    // checked that the ring still holds slot t).  The key of a token inside the
    // chunk comes from k_src.
    if (!early) {
      double2 hp[kSeg][NP], hq[kSeg][NP];
      RawD<T> kk[kSeg];
      int st_t[kSeg];
#pragma unroll
      for (int s = 0; s < kSeg; ++s) {
        const int ic = min(i0 + s, a.n_q - 1);
        int64_t t = past + ic - a.n_local;
        t = t < 0 ? 0 : t;
        const int sp = slot0 + ic - (slot0 + ic >= a.ring ? a.ring : 0);
        const int st = sp - a.n_local + (sp < a.n_local ? a.ring : 0);  // n_local < ring
        st_t[s] = st;
#pragma unroll
        for (int e = 0; e < NP; ++e) {
          hp[s][e] = ((const double2*)(ring + (int64_t)sp * D))[e];
          hq[s][e] = ((const double2*)(ring + (int64_t)st * D))[e];
        }
        kk[s] = t >= past
                    ? load_rawd<T>((const T*)a.k_src + (int64_t)bg * a.kv_head_stride + (t - past) * D + d0)
                    : load_rawd<T>(kread + ((int64_t)bg * a.capacity + t) * D + d0);
      }
#pragma unroll
      for (int s = 0; s < kSeg; ++s) {
        const int i = i0 + s;
        const int64_t t = past + i - a.n_local;
        const bool act = i < a.n_q && t >= a.n_init;
        float kt[kDPT];
        rawd_to_float<T>(kk[s], kt);
        if (ROPE) rotate_d(kt, t, d0 / 2, a.rope);  // the key at its own position, float32
        double p = 0.0;
#pragma unroll
        for (int e = 0; e < NP; ++e)
          p += (double)kt[2 * e] * (hp[s][e].x - hq[s][e].x) + (double)kt[2 * e + 1] * (hp[s][e].y - hq[s][e].y);
        p = add_halves(p);  // the two halves of the slice
        if (act && half == 0) a.rpart[((int64_t)bg * slices + slice) * a.ring + st_t[s]] = p;
      }
    }
  }
  if (qbar != nullptr && ROPE) {
    // plain query sum of the chunk: over the 32 segments of this half in the
    // wave, then over the waves
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) {
#pragma unroll
      for (int e = 0; e < kDPT; ++e) raw_acc[e] += __shfl_xor(raw_acc[e], o);
    }
    if ((lane & 31) == 0) {
#pragma unroll
      for (int e = 0; e < kDPT; ++e) wave_raw[wave][half][e] = raw_acc[e];
    }
    __syncthreads();
    if (seg == 0) {
#pragma unroll
      for (int e = 0; e < kDPT; ++e) {
        float t = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) t += wave_raw[w][half][e];
        qbar[(int64_t)bg * D + d0 + e] = t;
      }
    }
  } else if (qbar != nullptr && seg == 0) {
#pragma unroll
    for (int e = 0; e < kDPT; ++e) qbar[(int64_t)bg * D + d0 + e] = (float)(carry[e] - base[e]);
  }
}

}  // namespace

template <int DT>
static hipError_t launch_append_d(const AppendArgs& a, const BuildArgs& ba, const AppendGrid& g, hipStream_t s,
                                  float* qbar) {
  const int blocks = g.n_build + g.n_qsum + g.n_scan + g.n_copy_per_head * a.batch * a.n_kv_heads;
  if (blocks == 0) return hipSuccess;
  const dim3 grid(blocks);
  const int G = a.n_q_heads / a.n_kv_heads;
#define INFLLM_APPEND(T, GT)                                                                        \
  do {                                                                                             \
    if (a.rope.on)                                                                                 \
      hipLaunchKernelGGL((append_kernel<T, GT, DT, true>), grid, dim3(kThreads), 0, s, a, ba, g, qbar);  \
    else                                                                                           \
      hipLaunchKernelGGL((append_kernel<T, GT, DT, false>), grid, dim3(kThreads), 0, s, a, ba, g, qbar); \
  } while (0)
  if (a.bf16) {
    switch (G) {
      case 1: INFLLM_APPEND(bf16_t, 1); break;
      case 2: INFLLM_APPEND(bf16_t, 2); break;
      case 4: INFLLM_APPEND(bf16_t, 4); break;
      case 8: INFLLM_APPEND(bf16_t, 8); break;
      default: INFLLM_APPEND(bf16_t, 0); break;
    }
  } else {
    switch (G) {
      case 1: INFLLM_APPEND(float, 1); break;
      case 2: INFLLM_APPEND(float, 2); break;
      case 4: INFLLM_APPEND(float, 4); break;
      default: INFLLM_APPEND(float, 0); break;
    }
  }
#undef INFLLM_APPEND
  return hipGetLastError();
}

hipError_t launch_append(const AppendArgs& a, hipStream_t s, float* qbar, const BuildArgs* fused_build) {
  AppendGrid g;
  g.n_build = fused_build != nullptr ? fused_build->n_new * fused_build->batch * fused_build->n_kv_heads : 0;
  if (a.n_q == 0 && g.n_build == 0) return hipSuccess;
  const int esize = a.bf16 ? 2 : 4;
  g.thin = a.n_q <= kThinMaxQ;
  // The mean representation needs no query ring: copy (and build) blocks run, and
  // query-sum blocks when scoring follows (qbar given).
  g.qsum_parts = score_qbar_parts(a.n_q_heads / a.n_kv_heads, a.n_q);
  g.n_qsum = (a.mean_repr && qbar != nullptr && a.n_q > 0) ? g.qsum_parts * a.batch * a.n_kv_heads : 0;
  g.n_scan = (a.n_q <= 0 || a.mean_repr) ? 0
             : g.thin ? (a.batch * a.n_kv_heads * a.head_dim + kThreads - 1) / kThreads
                      : a.batch * a.n_kv_heads * (a.head_dim / kRpartDims);
  g.n_copy_per_head = 0;
  if (a.k_src != nullptr && a.n_q > 0) {
    const int vec_per_head = a.n_q * a.head_dim / (16 / esize);
    g.n_copy_per_head = (vec_per_head + kThreads * kCopyPerThread - 1) / (kThreads * kCopyPerThread);
  }
  BuildArgs ba;
  if (fused_build != nullptr) ba = *fused_build;
  else std::memset(&ba, 0, sizeof(ba));
  return a.head_dim == 128 ? launch_append_d<128>(a, ba, g, s, qbar) : launch_append_d<64>(a, ba, g, s, qbar);
}

}  // namespace infllm
