// bfloat16 attention for one current token per sequence (l_X = 1: decoding).
//
// With only G query rows per kv head the step streams the selected units, the
// initial and local tokens from HBM and does a few flops per byte, so the kernel
// is laid out for bandwidth: every wave-wide load moves whole key rows (one
// 16-byte piece per lane, D/8 lanes per key), each wave keeps the next two
// tiles' K and V rows in flight while it scores the current one, and the query
// rows of the group live in registers as bf16 pairs (8 dims per lane), so that
// the register budget leaves three waves per SIMD.  A q.k dot product is
// finished by a DPP all-reduce over the lanes of a key, so every lane of the key
// holds its score and reuses it as the weight of the same key's value piece.
//
// The virtual key axis of each (sequence, kv head) is split evenly into `parts`
// workgroups (the host picks enough parts to give every compute unit two
// workgroups), and each workgroup's keys evenly over its 4 waves, in whole
// tiles.  Each wave runs an online softmax over its keys, two tiles of loads
// ahead of the one it scores (running max raised only when a tile's max exceeds
// it by 2^8, so the common tile costs no rescale); the waves are combined
// through LDS into one partial result per workgroup, and the log-sum-exp merge
// of Section 3.1's split key set joins the workgroups.
#include "launch.h"

namespace infllm {
namespace {

constexpr int kDecodeWaves = 4;
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// v + (the value of v in the lanes given by the DPP control), one VALU op.
template <int CTRL>
__device__ __forceinline__ float dpp_add(float v) {
  return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ float dpp_max(float v) {
  return fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false)));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // lane i of each 8 <- lane 7-i
constexpr int kDppMirror = 0x140;      // lane i of each 16 <- lane 15-i
constexpr int kDppRor8 = 0x128;        // lane i of each 16 <- lane (i+8)%16

// Sum over the LPK lanes of one key (LPK = 8 or 16 consecutive lanes): after the
// two quad steps every quad holds its sum, the half mirror pairs quads 0|1 (and
// 2|3), the row mirror pairs the two halves of a row.
template <int LPK>
__device__ __forceinline__ float key_allreduce(float v) {
  v = dpp_add<kDppXor1>(v);
  v = dpp_add<kDppXor2>(v);
  v = dpp_add<kDppHalfMirror>(v);
  if constexpr (LPK == 16) v = dpp_add<kDppMirror>(v);
  return v;
}

// Sum / max over the key slots of a wave (the 64/LPK groups of LPK lanes): every
// lane ends with the value over all slots for its own lane-in-key index.
template <int LPK>
__device__ __forceinline__ float slots_sum(float v) {
  if constexpr (LPK == 8) v = dpp_add<kDppRor8>(v);
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
template <int LPK>
__device__ __forceinline__ float slots_max(float v) {
  if constexpr (LPK == 8) v = dpp_max<kDppRor8>(v);
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ __forceinline__ void bf16x8_to_f32(const uint4& raw, float (&f)[8]) {
  const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    f[2 * e] = __uint_as_float(w[e] << 16);
    f[2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
  }
}

constexpr uint32_t kNoKey = 0xFFFFFFFFu;

// Byte offset in the (sequence, kv head) slice of the store of the row of
// virtual key v, or kNoKey for a skipped unit entry.  The host guarantees that a
// slice spans less than 4 GiB, so 32-bit arithmetic is exact.  idx_row is the
// lookup row staged in LDS: reading it waits on the LDS counter only, never on
// the K/V loads in flight.
__device__ __forceinline__ uint32_t key_byte_offset(const StepGeom& g, const int32_t* idx_row, int v,
                                                    uint32_t row_bytes) {
  if (v < g.n_init) return (uint32_t)v * row_bytes;
  const int w = v - g.n_init;
  const int sel_len = g.n_sel * g.block_size;
  if (w < sel_len) {
    const int u = w / g.block_size;
    const int off = w - u * g.block_size;
    const int b = idx_row[u];
    if (b < 0 || b >= g.n_units) return kNoKey;
    return (uint32_t)(g.unit_base + b * g.block_size + off) * row_bytes;
  }
  return (uint32_t)(g.local_begin + (w - sel_len)) * row_bytes;
}

template <int D, int G>
__global__ void __launch_bounds__(64 * kDecodeWaves) attend_decode_kernel(AttendArgs a) {
  constexpr int LPK = D / 8;      // lanes per key row
  constexpr int KPI = 64 / LPK;   // keys per wave-wide load
  constexpr int NI = 2;           // K (and V) loads per lane per tile
  constexpr int TK = KPI * NI;    // keys per tile
  constexpr int NB = 3;           // tile buffers: two tiles in flight while one is scored

  __shared__ float cm[kDecodeWaves][G], cl[kDecodeWaves][G];
  __shared__ __attribute__((aligned(16))) float co[kDecodeWaves][G][D];
  __shared__ int32_t sidx[kDecodeMaxSel];
  __shared__ float fo[G][D];  // this part's output rows before the fp16 write

  const int part = blockIdx.x % a.parts;
  const int bg = blockIdx.x / a.parts;
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
  // this sequence's step (its own past length in a variable-length batch)
  const SeqStep sq = seq_step(a, b);
  const StepGeom& geo = sq.geom;
  const int mem_len = sq.mem_len, parts_mem = sq.parts_mem;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane % LPK, r = lane / LPK;  // 16-byte piece of the row, key slot of the load
  for (int j = tid; j < geo.n_sel; j += 64 * kDecodeWaves) sidx[j] = a.idx[(int64_t)bg * geo.idx_stride + j];

  // This wave's keys: the parts split the virtual axis evenly, in whole tiles per
  // wave.  With the positional remap parts [0, parts_mem) split the memory keys
  // [0, mem_len) (I and the units) and the other parts the local keys.
  const bool remap = a.rope.on != 0;
  const bool mem_part = part < parts_mem;
  int rv0 = 0, rv1 = geo.n_virtual, rpart = part, rparts = a.parts;
  if (mem_part) {
    rv1 = mem_len;
    rparts = parts_mem;
  } else if (parts_mem > 0) {
    rv0 = mem_len;
    rpart = part - parts_mem;
    rparts = a.parts - parts_mem;
  }
  const int n_waves_total = rparts * kDecodeWaves;
  const int kpw = ((rv1 - rv0 + n_waves_total - 1) / n_waves_total + TK - 1) / TK * TK;
  const int vw0 = rv0 + (rpart * kDecodeWaves + wave) * kpw;
  const int vw1 = min(vw0 + kpw, rv1);
  const int nt = vw1 > vw0 ? (vw1 - vw0 + TK - 1) / TK : 0;

  // Query rows of the group: this lane's 8 dims as 4 bf16 pairs; the dot products
  // take them as they are (v_dot2_f32_bf16) and are scaled by sm_scale * log2(e) after.
  const float c2 = a.sm_scale * 1.4426950408889634f;
  uint32_t qv[G][4];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const bf16_t* qp = (const bf16_t*)a.q + (int64_t)(b * a.n_q_heads + g * G + h) * a.q_head_stride + c * 8;
    const uint4 raw = *(const uint4*)qp;
    qv[h][0] = raw.x;
    qv[h][1] = raw.y;
    qv[h][2] = raw.z;
    qv[h][3] = raw.w;
  }
  if (remap) {
    // memory parts: the query turned by R(l_L); local parts: at its own position
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int pr = 4 * c + e;  // the pair held in word e
      float cs, sn;
      if (mem_part) {
        cs = a.rope.mem_cos[pr];
        sn = a.rope.mem_sin[pr];
      } else {
        rope_cos_sin(a.rope, geo.past_len, pr, cs, sn);
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float x0 = __uint_as_float(qv[h][e] << 16), x1 = __uint_as_float(qv[h][e] & 0xFFFF0000u);
        qv[h][e] = (uint32_t)f32_to_bf16(x0 * cs - x1 * sn) | ((uint32_t)f32_to_bf16(x0 * sn + x1 * cs) << 16);
      }
    }
  }
  __syncthreads();

  // uniform slice bases; per-lane 32-bit byte offsets (row offset + this lane's piece).
  // Local keys come rotated from k_rot under the remap.
  const char* kbase = (const char*)(remap && !mem_part ? a.k_rot : a.k_store) + (int64_t)bg * a.capacity * (D * 2);
  const char* vbase = (const char*)a.v_store + (int64_t)bg * a.capacity * (D * 2);
  const uint32_t piece = c * 16;

  uint4 kb[NB][NI], vb[NB][NI];
  bool valid[NB][NI];
  auto load_tile = [&](int t, int buf) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int v = vw0 + t * TK + i * KPI + r;
      const uint32_t o = v < vw1 ? key_byte_offset(geo, sidx, v, D * 2) : kNoKey;
      valid[buf][i] = o != kNoKey;
      const uint32_t oc = (o == kNoKey ? 0u : o) + piece;
      kb[buf][i] = *(const uint4*)(kbase + oc);
      vb[buf][i] = *(const uint4*)(vbase + oc);
    }
  };

  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -__builtin_inff();
    l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
  }

  auto consume = [&](int cur) {
    // scores of the tile's keys, every head of the group
    float s[G][NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const uint32_t kw[4] = {kb[cur][i].x, kb[cur][i].y, kb[cur][i].z, kb[cur][i].w};
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float d = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, qv[h][e]),
                                              __builtin_bit_cast(bf16x2_t, kw[e]), d, false);
        s[h][i] = d;
      }
    }
    float mx[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      mx[h] = -__builtin_inff();
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        s[h][i] = valid[cur][i] ? key_allreduce<LPK>(s[h][i]) * c2 : -__builtin_inff();
        mx[h] = fmaxf(mx[h], s[h][i]);
      }
      mx[h] = slots_max<LPK>(mx[h]);
    }
    // lazy running max (the decision is wave-uniform)
    bool grow = false;
#pragma unroll
    for (int h = 0; h < G; ++h) grow |= mx[h] > m[h] + 8.f;
    if (grow) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float m_new = fmaxf(m[h], mx[h]);
        const float sc = m[h] == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(m[h] - m_new);
        m[h] = m_new;
        l[h] *= sc;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] *= sc;
      }
    }
    // weights and the value pieces (a key with no row contributes exactly 0)
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      float vf[8];
      bf16x8_to_f32(vb[cur][i], vf);
#pragma unroll
      for (int e = 0; e < 8; ++e) vf[e] = valid[cur][i] ? vf[e] : 0.f;
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float base = m[h] == -__builtin_inff() ? 0.f : m[h];
        const float p = __builtin_amdgcn_exp2f(s[h][i] - base);
        l[h] += p;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] += p * vf[e];
      }
    }
  };

  // NB-deep pipeline over the wave's tiles (buffer of tile t: t % NB).  The tile
  // count is padded to a multiple of NB and every load is issued unconditionally
  // (tiles past the end read row 0 and count as empty), so no branch separates a
  // load from its use and the load counter waits only for the tile at hand.
  const int nt_pad = (nt + NB - 1) / NB * NB;
#pragma unroll
  for (int t = 0; t < NB - 1; ++t) load_tile(t, t);
  for (int t0 = 0; t0 < nt_pad; t0 += NB) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      load_tile(t0 + j + NB - 1, (j + NB - 1) % NB);
      consume(j);
    }
  }

  // Wave totals: sum the key slots; the lanes of slot 0 hold the wave's result.
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float lt = slots_sum<LPK>(l[h]);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = slots_sum<LPK>(acc[h][e]);
    if (r == 0) {
      *(float4*)&co[wave][h][c * 8] = make_float4(acc[h][0], acc[h][1], acc[h][2], acc[h][3]);
      *(float4*)&co[wave][h][c * 8 + 4] = make_float4(acc[h][4], acc[h][5], acc[h][6], acc[h][7]);
    }
    if (lane == 0) {
      cm[wave][h] = m[h];
      cl[wave][h] = lt;
    }
  }
  __syncthreads();

  // Combine the waves (exp2 domain).  One part: write the bf16 output directly.
  // Several: stage the part's rows in LDS, then each wave writes whole rows as
  // fp16 scaled by their per-row exponent.
  const int64_t rows_total = (int64_t)a.batch * a.n_q_heads;  // n_q == 1
  for (int e = tid; e < G * D; e += 64 * kDecodeWaves) {
    const int h = e / D, d = e - h * D;
    float M = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < kDecodeWaves; ++w) M = fmaxf(M, cm[w][h]);
    float L = 0.f, O = 0.f;
    if (M != -__builtin_inff()) {
#pragma unroll
      for (int w = 0; w < kDecodeWaves; ++w) {
        const float wt = cm[w][h] == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(cm[w][h] - M);
        L += wt * cl[w][h];
        O += wt * co[w][h][d];
      }
    }
    const float o = L > 0.f ? O / L : 0.f;
    const int64_t grow_ = (int64_t)b * a.n_q_heads + g * G + h;
    if (a.parts == 1) ((bf16_t*)a.out)[grow_ * a.out_head_stride + d] = f32_to_bf16(o);
    else fo[h][d] = o;
    if (d == 0) {
      const float lse_v = L > 0.f ? (M + __log2f(L)) * 0.6931471805599453f : -__builtin_inff();
      if (a.parts == 1) {
        if (a.lse != nullptr) a.lse[grow_] = lse_v;
      } else {
        a.part_lse[(int64_t)part * rows_total + grow_] = lse_v;
      }
    }
  }
  if (a.parts == 1) return;
  __syncthreads();
  constexpr int PL = D / 64;  // values per lane of a row
  for (int h = wave; h < G; h += kDecodeWaves) {
    float v[PL];
    float amax = 0.f;
#pragma unroll
    for (int j = 0; j < PL; ++j) {
      v[j] = fo[h][lane * PL + j];
      amax = fmaxf(amax, fabsf(v[j]));
    }
    const int ex = partial_row_exponent(wave_max(amax));
    const float sc = exp2_int(-ex);
    const int64_t grow_ = (int64_t)b * a.n_q_heads + g * G + h;
    uint16_t* op = (uint16_t*)a.part_o + ((int64_t)part * rows_total + grow_) * D + lane * PL;
    if constexpr (PL == 2) {
      *(uint32_t*)op = pack_f16x2(v[0] * sc, v[1] * sc);
    } else {
      const _Float16 hv = (_Float16)(v[0] * sc);
      *op = __builtin_bit_cast(uint16_t, hv);
    }
    if (lane == 0) a.part_exp[(int64_t)part * rows_total + grow_] = ex;
  }
}

template <int D>
hipError_t launch_decode_d(const AttendArgs& a, hipStream_t s) {
  const int G = a.n_q_heads / a.n_kv_heads;
  const dim3 grid(a.parts * a.batch * a.n_kv_heads), block(64 * kDecodeWaves);
  switch (G) {
    case 1: hipLaunchKernelGGL((attend_decode_kernel<D, 1>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((attend_decode_kernel<D, 2>), grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL((attend_decode_kernel<D, 4>), grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL((attend_decode_kernel<D, 8>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attend_decode(const AttendArgs& a, hipStream_t s) {
  return a.head_dim == 128 ? launch_decode_d<128>(a, s) : launch_decode_d<64>(a, s);
}

}  // namespace infllm
