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

// Stored column of key `key` (0..63) in a V^T row: groups of 16 keys, each group
// ordered [0-3, 8-11, 4-7, 12-15].
__device__ __forceinline__ int vt_col(int key) {
  const int k16 = key & 15;
  return (key & ~15) + 8 * ((k16 >> 2) & 1) + 4 * (k16 >> 3) + (k16 & 3);
}

template <int D>
struct Smem {
  static constexpr int KP = D + 8;   // K row pitch (bf16)
  static constexpr int VP = KB + 8;  // V^T row pitch (bf16)
  bf16_t k[2][KB * KP];
  bf16_t vt[2][D * VP];
  uint8_t kvalid[2][KB];
  int has_invalid;
};

template <int D>
__global__ void __launch_bounds__(256, 2) attend_mfma_kernel(AttendArgs a) {
  constexpr int KP = Smem<D>::KP, VP = Smem<D>::VP;
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
      uint4 raw = row_ok ? *(const uint4*)(qp + 16 * s + 8 * gsel) : make_uint4(0, 0, 0, 0);
      qreg[s] = __builtin_bit_cast(bf16x8, raw);
    }
  }

  // Staging: each thread moves 4 consecutive keys x 8 dims of K and of V.
  constexpr int PATCHES = (KB / 4) * CH;
  constexpr int PPT = (PATCHES + 255) / 256;
  uint4 kreg[PPT][4], vreg[PPT][4];
  uint8_t vmask[PPT];

  auto load_tile = [&](int tile) {
#pragma unroll
    for (int pp = 0; pp < PPT; ++pp) {
      const int p = tid + pp * 256;
      vmask[pp] = 0;
      if (p < PATCHES) {
        const int kq = p / CH, c = p - (p / CH) * CH;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int v = tile * KB + 4 * kq + i;
          const int64_t pos = (v < geo.n_virtual) ? virtual_pos(geo, idx_row, v) : -1;
          if (pos >= 0) {
            kreg[pp][i] = *(const uint4*)(kbase + pos * D + 8 * c);
            vreg[pp][i] = *(const uint4*)(vbase + pos * D + 8 * c);
            vmask[pp] |= (uint8_t)(1u << i);
          } else {
            kreg[pp][i] = make_uint4(0, 0, 0, 0);
            vreg[pp][i] = make_uint4(0, 0, 0, 0);
          }
        }
      }
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int pp = 0; pp < PPT; ++pp) {
      const int p = tid + pp * 256;
      if (p < PATCHES) {
        const int kq = p / CH, c = p - (p / CH) * CH;
#pragma unroll
        for (int i = 0; i < 4; ++i) *(uint4*)(&sm.k[buf][(4 * kq + i) * KP + 8 * c]) = kreg[pp][i];
        const int col = vt_col(4 * kq);
#pragma unroll
        for (int w = 0; w < 4; ++w) {  // dword w of the 16-byte chunk = dims 8c+2w, 8c+2w+1
          const uint32_t k0 = ((const uint32_t*)&vreg[pp][0])[w], k1 = ((const uint32_t*)&vreg[pp][1])[w];
          const uint32_t k2 = ((const uint32_t*)&vreg[pp][2])[w], k3 = ((const uint32_t*)&vreg[pp][3])[w];
          uint2 lo, hi;  // lo: dim 2w for keys 0..3, hi: dim 2w+1
          lo.x = (k0 & 0xFFFFu) | (k1 << 16);
          lo.y = (k2 & 0xFFFFu) | (k3 << 16);
          hi.x = (k0 >> 16) | (k1 & 0xFFFF0000u);
          hi.y = (k2 >> 16) | (k3 & 0xFFFF0000u);
          *(uint2*)(&sm.vt[buf][(8 * c + 2 * w) * VP + col]) = lo;
          *(uint2*)(&sm.vt[buf][(8 * c + 2 * w + 1) * VP + col]) = hi;
        }
        if (c == 0) {
#pragma unroll
          for (int i = 0; i < 4; ++i) sm.kvalid[buf][4 * kq + i] = (vmask[pp] >> i) & 1u;
        }
      }
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
    store_tile(0);
  }
  __syncthreads();
  const bool has_invalid = sm.has_invalid != 0;

  for (int t = t_begin; t < t_end; ++t) {
    const int buf = (t - t_begin) & 1;
    if (t + 1 < t_end) load_tile(t + 1);

    const bf16_t* Kb = sm.k[buf];
    const bf16_t* Vb = sm.vt[buf];
    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int j = 0; j < 16; ++j) sacc[kb][j] = 0.f;
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
        const bf16x8 ka = *(const bf16x8*)(Kb + (32 * kb + n) * KP + 16 * s + 8 * gsel);
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qreg[s], sacc[kb], 0, 0, 0);
      }
    }

    // Masks: current tokens (causal), the ragged end, skipped unit entries.
    const int tile_v0 = t * KB;
    const bool need_mask = (tile_v0 + KB > v_x0) || has_invalid;
    float mx = -__builtin_inff();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        float x = sacc[kb][j] * c2;
        if (need_mask) {
          const int kl = 32 * kb + 8 * (j >> 2) + 4 * gsel + (j & 3);
          const int v = tile_v0 + kl;
          const bool vis = sm.kvalid[buf][kl] && v < geo.n_virtual && (v < v_x0 || v - v_x0 <= qi);
          x = vis ? x : -__builtin_inff();
        }
        sacc[kb][j] = x;
        mx = fmaxf(mx, x);
      }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float base = (m_new == -__builtin_inff()) ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - base);
    float psum = 0.f;
    bf16x8 pb[2][2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float p = fast_exp2(sacc[kb][j] - base);
        psum += p;
        pb[kb][j >> 3][j & 7] = (__bf16)p;
      }
    }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) oacc[db][j] *= alpha;

#pragma unroll
    for (int db = 0; db < DBLK; ++db) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const bf16x8 va = *(const bf16x8*)(Vb + (32 * db + n) * VP + 16 * (2 * kb + h) + 8 * gsel);
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[kb][h], oacc[db], 0, 0, 0);
        }
      }
    }

    if (t + 1 < t_end) store_tile(buf ^ 1);
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
