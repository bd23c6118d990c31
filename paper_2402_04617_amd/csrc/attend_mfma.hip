// Chunk attention over Concat(I, selected units, L, X) (Section 3.1) in bf16 on
// CDNA4 matrix cores (v_mfma_f32_32x32x16_bf16), fp32 accumulation.
//
// Work decomposition
//   rows   : per (sequence, kv head) the G*n_q query rows (row r -> query i = r/G,
//            head g*G + r%G), so the G heads sharing a K/V tile are packed together;
//            128 rows per workgroup, 32 per wave.
//   keys   : the virtual key axis (see StepGeom) in tiles of 64 keys, gathered
//            straight from the token-ordered store (a selected unit is contiguous),
//            double-buffered through LDS; optionally split into parts whose partial
//            softmaxes are merged afterwards by log-sum-exp.
// Per wave and key tile:
//   S^T = K Q^T  : A = K tile rows from LDS, B = the wave's Q rows held in VGPRs.
//                  The 32x32 accumulator gives each lane one query row and 16 keys.
//   online softmax in the exp2 domain, row max combined across the two lane halves.
//   O^T += V^T P^T: B = P^T taken directly from the S^T accumulator (no shuffle);
//                  A = V^T from LDS, where V is stored transposed with the key order
//                  inside each 16-key group permuted to match the accumulator's key
//                  order, so each A fragment is one 16-byte LDS read.
#include "launch.h"

namespace infllm {
namespace {

constexpr int KB = 64;      // keys per tile
constexpr int NWAVE = 4;
constexpr int ROWS_WG = 32 * NWAVE;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ uint32_t dword(const u32x4& v, int w) { return v[w]; }

// Stored column of key `key` (0..63) in a V^T row: groups of 16 keys, each group
// ordered [0-3, 8-11, 4-7, 12-15].
__device__ __forceinline__ int vt_col(int key) {
  const int k16 = key & 15;
  return (key & ~15) + 8 * ((k16 >> 2) & 1) + 4 * (k16 >> 3) + (k16 & 3);
}

struct Stage {
  u32x4 k0, k1, k2, k3, v0, v1, v2, v3;
  uint32_t mask;
};

// LDS tiles are unpadded and XOR-swizzled at 16-byte (8 x bf16) granularity, so
// that both the MFMA fragment reads (8 consecutive rows, one granule each) and
// the staging writes spread over all LDS banks.
//   K   [64 keys][D]:  granule g of row r stored at g ^ (r & 7)
//   V^T [D][64 keys]:  granule g of row r stored at g ^ ((r & 7) ^ ((r >> 3) & 7))
template <int D>
__device__ __forceinline__ int k_lds(int r, int g) { return r * D + 8 * (g ^ (r & 7)); }
__device__ __forceinline__ int vt_lds(int r, int g) { return r * KB + 8 * (g ^ ((r & 7) ^ ((r >> 3) & 7))); }

template <int D>
struct Smem {
  bf16_t k[2][KB * D];
  bf16_t vt[2][D * KB];
  uint8_t kvalid[2][KB];
  int has_invalid;
};

template <int D>
__global__ void __launch_bounds__(256, 2) attend_mfma_kernel(AttendArgs a) {
  constexpr int CH = D / 8;      // 16-byte chunks per row
  constexpr int KSTEPS = D / 16; // MFMA k-steps over the head dim
  constexpr int DBLK = D / 32;   // 32-wide output blocks
  __shared__ __attribute__((aligned(16))) Smem<D> sm;

  const StepGeom& geo = a.geom;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int R = G * geo.n_q;
  const int n_row_tiles = (R + ROWS_WG - 1) / ROWS_WG;
  const int L = xcd_logical_block(blockIdx.x, gridDim.x);
  const int rt = L % n_row_tiles;
  const int tmp = L / n_row_tiles;
  const int part = tmp % a.parts;
  const int bg = tmp / a.parts;
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;

  const int n_tiles = (geo.n_virtual + KB - 1) / KB;
  const int per_part = (n_tiles + a.parts - 1) / a.parts;
  const int t_begin = part * per_part;
  int t_end = min(n_tiles, t_begin + per_part);
  const int v_x0 = geo.n_virtual - geo.n_q;  // first current-token key
  {
    const int i_max = (min(R, (rt + 1) * ROWS_WG) - 1) / G;
    t_end = min(t_end, (v_x0 + i_max) / KB + 1);  // tiles past this are fully causal-masked
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, gsel = lane >> 5;
  const int row = rt * ROWS_WG + wave * 32 + n;
  const bool row_ok = row < R;
  const int qi = row_ok ? row / G : 0;
  const int qh = g * G + (row_ok ? row - qi * G : 0);

  const int32_t* idx_row = a.idx + (int64_t)bg * geo.idx_stride;
  const bf16_t* kbase = (const bf16_t*)a.k_store + (int64_t)bg * a.capacity * D;
  const bf16_t* vbase = (const bf16_t*)a.v_store + (int64_t)bg * a.capacity * D;

  if (tid == 0) {
    int bad = 0;
    for (int u = 0; u < geo.n_sel; ++u) bad |= (idx_row[u] < 0 || idx_row[u] >= geo.n_units);
    sm.has_invalid = bad;
  }

  // Q rows of this wave as the B operand (8 bf16 per lane per k-step).
  bf16x8 qreg[KSTEPS];
  {
    const bf16_t* qp = (const bf16_t*)a.q + (int64_t)(b * a.n_q_heads + qh) * a.q_head_stride + (int64_t)qi * D;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      const u32x4 raw = row_ok ? *(const u32x4*)(qp + 16 * s + 8 * gsel) : u32x4{0, 0, 0, 0};
      qreg[s] = __builtin_bit_cast(bf16x8, raw);
    }
  }

  // Staging: each thread moves 4 consecutive keys x 8 dims of K and of V (one
  // patch; for D = 64 half the threads idle).
  constexpr int PATCHES = (KB / 4) * CH;
  static_assert(PATCHES <= 256, "one patch per thread");
  const bool stager = tid < PATCHES;
  const int kq = (tid % PATCHES) / CH, kc = tid % CH;  // non-stagers load a duplicate patch, store nothing
  Stage st;

  // A tile inside one segment (I, one selected unit, or the L+X run) maps to 64
  // consecutive store positions: the common case, gathered with no per-key work.
  // Returns that first position (uniform across the workgroup) or -1.
  auto tile_run_start = [&](int tile) -> int64_t {
    const int v0 = tile * KB;
    if (v0 + KB > geo.n_virtual) return -1;
    if (v0 + KB <= geo.n_init) return v0;
    if (v0 < geo.n_init) return -1;
    const int w = v0 - geo.n_init;
    const int sel_len = geo.n_sel * geo.block_size;
    if (w >= sel_len) return geo.local_begin + (w - sel_len);
    if (w + KB > sel_len) return -1;
    const int u = w / geo.block_size;
    if ((w + KB - 1) / geo.block_size != u) return -1;
    const int bu = idx_row[u];
    if (bu < 0 || bu >= geo.n_units) return -1;
    return (int64_t)geo.unit_base + (int64_t)bu * geo.block_size + (w - u * geo.block_size);
  };

  // Both gather paths only produce positions; the loads themselves are common,
  // unconditional and branch-free.  A key that is not part of the context
  // (ragged end, skipped unit entry) reads position 0 -- always written -- and is
  // masked to -inf before the softmax, so its (finite) K/V never contribute.
  auto load_tile = [&](int tile) {
    const int64_t r = tile_run_start(tile);  // uniform: keep it in scalar registers
    const int64_t run0 = ((int64_t)__builtin_amdgcn_readfirstlane((int)(r >> 32)) << 32) |
                         (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)r);
    int64_t p0, p1, p2, p3;
    if (run0 >= 0) {
      st.mask = 0xF;
      p0 = run0 + 4 * kq;
      p1 = p0 + 1;
      p2 = p0 + 2;
      p3 = p0 + 3;
    } else {
      const int v = tile * KB + 4 * kq;
      const int64_t q0 = (v + 0 < geo.n_virtual) ? virtual_pos(geo, idx_row, v + 0) : -1;
      const int64_t q1 = (v + 1 < geo.n_virtual) ? virtual_pos(geo, idx_row, v + 1) : -1;
      const int64_t q2 = (v + 2 < geo.n_virtual) ? virtual_pos(geo, idx_row, v + 2) : -1;
      const int64_t q3 = (v + 3 < geo.n_virtual) ? virtual_pos(geo, idx_row, v + 3) : -1;
      st.mask = (q0 >= 0 ? 1u : 0u) | (q1 >= 0 ? 2u : 0u) | (q2 >= 0 ? 4u : 0u) | (q3 >= 0 ? 8u : 0u);
      p0 = q0 >= 0 ? q0 : 0;
      p1 = q1 >= 0 ? q1 : 0;
      p2 = q2 >= 0 ? q2 : 0;
      p3 = q3 >= 0 ? q3 : 0;
    }
    st.k0 = *(const u32x4*)(kbase + p0 * D + 8 * kc);
    st.k1 = *(const u32x4*)(kbase + p1 * D + 8 * kc);
    st.k2 = *(const u32x4*)(kbase + p2 * D + 8 * kc);
    st.k3 = *(const u32x4*)(kbase + p3 * D + 8 * kc);
    st.v0 = *(const u32x4*)(vbase + p0 * D + 8 * kc);
    st.v1 = *(const u32x4*)(vbase + p1 * D + 8 * kc);
    st.v2 = *(const u32x4*)(vbase + p2 * D + 8 * kc);
    st.v3 = *(const u32x4*)(vbase + p3 * D + 8 * kc);
  };
  // The buffer of tile t+1 is not read during iteration t (the barrier ending
  // iteration t-1 retired its last readers), so K and V are written into it as
  // soon as convenient, which keeps their staging registers short-lived.
  auto store_k = [&](int buf) {
    if (!stager) return;
    bf16_t* kd = sm.k[buf];
    *(u32x4*)(kd + k_lds<D>(4 * kq + 0, kc)) = st.k0;
    *(u32x4*)(kd + k_lds<D>(4 * kq + 1, kc)) = st.k1;
    *(u32x4*)(kd + k_lds<D>(4 * kq + 2, kc)) = st.k2;
    *(u32x4*)(kd + k_lds<D>(4 * kq + 3, kc)) = st.k3;
  };
  auto store_v = [&](int buf) {
    if (!stager) return;
    const int col = vt_col(4 * kq);        // logical column of the 4-key run in a V^T row
    const int g = col >> 3, half = (col >> 2) & 1;
    bf16_t* vd = sm.vt[buf];
#pragma unroll
    for (int w = 0; w < 4; ++w) {  // dword w of the 16-byte chunk = dims 8c+2w, 8c+2w+1
      const uint32_t a0 = dword(st.v0, w), a1 = dword(st.v1, w);
      const uint32_t a2 = dword(st.v2, w), a3 = dword(st.v3, w);
      uint2 lo, hi;  // lo: dim 2w for keys 0..3, hi: dim 2w+1
      lo.x = (a0 & 0xFFFFu) | (a1 << 16);
      lo.y = (a2 & 0xFFFFu) | (a3 << 16);
      hi.x = (a0 >> 16) | (a1 & 0xFFFF0000u);
      hi.y = (a2 >> 16) | (a3 & 0xFFFF0000u);
      const int r = 8 * kc + 2 * w;
      *(uint2*)(vd + vt_lds(r, g) + 4 * half) = lo;
      *(uint2*)(vd + vt_lds(r + 1, g) + 4 * half) = hi;
    }
    if (kc == 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i) sm.kvalid[buf][4 * kq + i] = (st.mask >> i) & 1u;
    }
  };

  f32x16 oacc[DBLK];
#pragma unroll
  for (int db = 0; db < DBLK; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) oacc[db][j] = 0.f;
  float m_run = -__builtin_inff();
  float l_run = 0.f;
  const float c2 = a.sm_scale * 1.4426950408889634f;

  if (t_begin < t_end) {
    load_tile(t_begin);
    store_k(0);
    store_v(0);
  }
  __syncthreads();
  const bool has_invalid = sm.has_invalid != 0;

  // Loop-invariant per-lane LDS offsets (elements) of the MFMA fragments under
  // the swizzles: K k-steps 4..7 repeat k-steps 0..3 one 64-element half-row
  // further; V^T offsets depend only on the parity of the 32-row block.
  int koff[4], voff[2][4];
#pragma unroll
  for (int s = 0; s < 4; ++s) koff[s] = n * D + 8 * ((2 * s + gsel) ^ (n & 7));
#pragma unroll
  for (int par = 0; par < 2; ++par)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      voff[par][j] = n * KB + 8 * ((2 * j + gsel) ^ ((n & 7) ^ (((n >> 3) + 4 * par) & 7)));

  for (int t = t_begin; t < t_end; ++t) {
    const int buf = (t - t_begin) & 1;
    // Unconditional prefetch (the last iteration re-fetches its own tile and
    // never stores it): no register join at the back edge, so the loads stay
    // in flight across the whole iteration.
    load_tile(min(t + 1, t_end - 1));

    const bf16_t* Kb = sm.k[buf];
    const bf16_t* Vb = sm.vt[buf];
    // S^T for keys [0,32) and [32,64) of the tile: two independent accumulator
    // chains interleaved, K fragments read two k-steps ahead of their MFMA.
    f32x16 sacc[2];
    {
      // lane (n, gsel) reads row 32*kb + n, granule 2*s + gsel (swizzled by n & 7)
      const bf16_t* kr0 = Kb;
      const bf16_t* kr1 = Kb + 32 * D;
      auto kfrag = [&](const bf16_t* base, int s) {
        return *(const bf16x8*)(base + koff[s & 3] + 64 * (s >> 2));
      };
      bf16x8 a0[2], a1[2];
      a0[0] = kfrag(kr0, 0);
      a1[0] = kfrag(kr1, 0);
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
        if (s + 1 < KSTEPS) {
          a0[(s + 1) & 1] = kfrag(kr0, s + 1);
          a1[(s + 1) & 1] = kfrag(kr1, s + 1);
        }
        if (s == 0) {
          const f32x16 zero = {};
          sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[0], qreg[0], zero, 0, 0, 0);
          sacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[0], qreg[0], zero, 0, 0, 0);
        } else {
          sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[s & 1], qreg[s], sacc[0], 0, 0, 0);
          sacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[s & 1], qreg[s], sacc[1], 0, 0, 0);
        }
      }
    }
    // lane (n, gsel) reads V^T row 32*db + n, granule 2*j + gsel of P block j
    auto vfrag = [&](int db, int j) { return *(const bf16x8*)(Vb + 32 * db * KB + voff[db & 1][j]); };

    // Masks: current tokens (causal), the ragged end, skipped unit entries.
    const int tile_v0 = t * KB;
    const bool need_mask = (tile_v0 + KB > v_x0) || has_invalid;
    float mx = -__builtin_inff();
    if (need_mask) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int kl = 32 * kb + 8 * (j >> 2) + 4 * gsel + (j & 3);
          const int v = tile_v0 + kl;
          const bool vis = sm.kvalid[buf][kl] && v < geo.n_virtual && (v < v_x0 || v - v_x0 <= qi);
          sacc[kb][j] = vis ? sacc[kb][j] : -__builtin_inff();
        }
      }
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 16; ++j) mx = fmaxf(mx, sacc[kb][j]);
    mx = fmaxf(mx, __shfl_xor(mx, 32)) * c2;  // row max of this tile, in the exp2 domain (c2 > 0)

    // Rescale only when some row's max grew by more than 2^8 since the last
    // rescale; otherwise keep the stale max (p <= 256, exact after the final
    // normalisation).  The decision is wave-uniform, so both lane halves of a
    // row always use the same max.
    if (__ballot(mx > m_run + 8.f)) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = (m_new == -__builtin_inff()) ? 1.f : fast_exp2(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DBLK; ++db)
#pragma unroll
        for (int j = 0; j < 16; ++j) oacc[db][j] *= alpha;
      m_run = m_new;
    }
    const float neg_m = (m_run == -__builtin_inff()) ? 0.f : -m_run;
    float psum = 0.f;
    bf16x8 pb[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float p = fast_exp2(__builtin_fmaf(sacc[kb][j], c2, neg_m));
        psum += p;
        pb[kb][j >> 3][j & 7] = (__bf16)p;
      }
    }
    l_run += psum;

    bf16x8 va[DBLK];
#pragma unroll
    for (int db = 0; db < DBLK; ++db) va[db] = vfrag(db, 0);
    if (t + 1 < t_end) store_k(buf ^ 1);

    // O^T += V^T P^T over the four 16-key blocks of P; DBLK independent
    // accumulator chains per block, each fragment register refilled with the
    // next block's fragment right after the MFMA that consumed it.
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int db = 0; db < DBLK; ++db) {
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[db], pb[j >> 1][j & 1], oacc[db], 0, 0, 0);
        if (j + 1 < 4) va[db] = vfrag(db, j + 1);
      }
    }

    if (t + 1 < t_end) store_v(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: combine the two lane halves' partial sums; write O and lse.
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_v = (m_run == -__builtin_inff() || l_tot <= 0.f)
                          ? -__builtin_inff()
                          : (m_run + __log2f(l_tot)) * 0.6931471805599453f;
  if (!row_ok) return;
  const int64_t grow = ((int64_t)(b * a.n_q_heads + qh)) * geo.n_q + qi;
  if (a.parts == 1) {
    bf16_t* op = (bf16_t*)a.out + (int64_t)(b * a.n_q_heads + qh) * a.out_head_stride + (int64_t)qi * D;
#pragma unroll
    for (int db = 0; db < DBLK; ++db) {
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int d = 32 * db + 8 * jq + 4 * gsel;
        uint2 w;
        w.x = (uint32_t)f32_to_bf16(oacc[db][4 * jq] * inv) | ((uint32_t)f32_to_bf16(oacc[db][4 * jq + 1] * inv) << 16);
        w.y = (uint32_t)f32_to_bf16(oacc[db][4 * jq + 2] * inv) | ((uint32_t)f32_to_bf16(oacc[db][4 * jq + 3] * inv) << 16);
        *(uint2*)(op + d) = w;
      }
    }
    if (a.lse != nullptr && gsel == 0) a.lse[grow] = lse_v;
  } else {
    const int64_t rows_total = (int64_t)a.batch * a.n_q_heads * geo.n_q;
    float* op = a.part_o + ((int64_t)part * rows_total + grow) * D;
#pragma unroll
    for (int db = 0; db < DBLK; ++db) {
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int d = 32 * db + 8 * jq + 4 * gsel;
        *(float4*)(op + d) = make_float4(oacc[db][4 * jq] * inv, oacc[db][4 * jq + 1] * inv,
                                         oacc[db][4 * jq + 2] * inv, oacc[db][4 * jq + 3] * inv);
      }
    }
    if (gsel == 0) a.part_lse[(int64_t)part * rows_total + grow] = lse_v;
  }
}

}  // namespace

hipError_t launch_attend_mfma(const AttendArgs& a, hipStream_t s) {
  const int G = a.n_q_heads / a.n_kv_heads;
  const int R = G * a.geom.n_q;
  const int n_row_tiles = (R + ROWS_WG - 1) / ROWS_WG;
  const int blocks = n_row_tiles * a.parts * a.batch * a.n_kv_heads;
  if (a.head_dim == 128)
    hipLaunchKernelGGL(attend_mfma_kernel<128>, dim3(blocks), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(attend_mfma_kernel<64>, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace infllm
