// Attention mass of the looked-up memory units and the decayed frequency score
// (Section 3.2, "Cache Management"; the appendix on the cache-management
// strategy).  For kv head g and looked-up unit b the mass is the softmax
// probability that the step's attention gave the unit's l_bs keys, summed over
// the chunk's queries and the G query heads of the group:
//   mass(b) = sum_h sum_i sum_{t in b} exp(z^h_i(t) - lse^h_i),
// with z the attention logit (sm_scale * q . k; under the positional remap the
// query turned by R(l_L), as for every memory key) and lse the step's final
// natural-log normaliser.  The frequency score of every built unit then decays,
// s_b <- s_b * d, and a looked-up unit adds its mass.
//
// One workgroup (16 waves) per (sequence*kv head, lookup slot).  bf16: the unit's
// keys are staged in LDS once (rows padded by 16 bytes so the fragment reads of
// 32 rows spread over the banks); each wave takes two 32-row blocks of the
// group's queries at a time as B operands of v_mfma_f32_32x32x16_bf16, so every
// K fragment read from LDS (one k-step ahead) feeds two independent accumulator
// chains; each score is exponentiated against its row's lse and summed, one
// float per lane, then a wave and a workgroup sum.  float32: plain dot products
// per (row, key).  Extra workgroups, one per (sequence*kv head), decay the scores
// of the units not looked up, so every score is written by exactly one thread.
#include "launch.h"

namespace infllm {
namespace {

constexpr int kMassThreads = 1024;
constexpr int kMassWaves = kMassThreads / 64;
constexpr int kMassMaxBlock = 256;  // largest l_bs

// Sum of a float over a workgroup of NW waves (every thread gets it).
template <int NW = kMassWaves>
__device__ __forceinline__ float block_sum(float x, float* red) {
  x = wave_sum(x);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = x;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int w = 0; w < NW; ++w) t += red[w];
  return t;
}

// Decay of the frequency scores of the units that row's lookup idx_row did not
// take (the looked-up ones are updated by their slot's workgroup, so every score
// is written by exactly one thread).
// Scores are read BATCH per thread at a time, every load before the first store;
// the looked-up units are marked in an LDS bitmap first (one lookup per unit
// instead of a scan of the row's k entries).
constexpr int kDecayBitmapWords = 2048;  // units 0 .. 65,535
template <int BATCH>
__device__ void decay_unselected(const int32_t* idx_row, int k, float* f, int n_units, float decay, int* sel) {
  __shared__ uint32_t bits[kDecayBitmapWords];
  const int step = blockDim.x;
  const bool bitmap = n_units <= 32 * kDecayBitmapWords;
  // the first batch of scores is in flight while the lookup row is marked
  float fv[BATCH];
#pragma unroll
  for (int i = 0; i < BATCH; ++i) {
    const int u = threadIdx.x + i * step;
    fv[i] = f[min(u, n_units - 1)];
  }
  if (bitmap) {
    for (int w = threadIdx.x; w < (n_units + 31) / 32; w += step) bits[w] = 0u;
    __syncthreads();
    for (int j = threadIdx.x; j < k; j += step) {
      const int u = idx_row[j];
      if (u >= 0 && u < n_units) atomicOr(&bits[u >> 5], 1u << (u & 31));
    }
  } else {
    for (int j = threadIdx.x; j < k; j += step) sel[j] = idx_row[j];
  }
  __syncthreads();
  for (int u0 = threadIdx.x; u0 < n_units; u0 += step * BATCH) {
    if (u0 != (int)threadIdx.x) {
#pragma unroll
      for (int i = 0; i < BATCH; ++i) fv[i] = f[min(u0 + i * step, n_units - 1)];
    }
#pragma unroll
    for (int i = 0; i < BATCH; ++i) {
      const int u = u0 + i * step;
      if (u >= n_units) continue;
      bool looked_up = false;
      if (bitmap) {
        looked_up = ((bits[u >> 5] >> (u & 31)) & 1u) != 0u;
      } else {
        for (int j = 0; j < k; ++j) looked_up |= sel[j] == u;
      }
      if (!looked_up) f[u] = fv[i] * decay;
    }
  }
}

// Mass of one looked-up unit, bf16 inputs (D = 64 or 128).
template <int D>
__device__ void unit_mass_bf16(const MassArgs& a, int bg, int slot, int unit, float* red) {
  constexpr int KSTEPS = D / 16;
  constexpr int ROW_BYTES = D * 2 + 16;  // padded LDS row
  __shared__ __attribute__((aligned(16))) uint8_t ks[kMassMaxBlock * ROW_BYTES];
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int lbs = a.block_size;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // the unit's keys -> LDS (unrotated: memory keys)
  const bf16_t* kb = (const bf16_t*)a.k_store + ((int64_t)bg * a.capacity + a.n_init + (int64_t)unit * lbs) * D;
  for (int e = tid; e < lbs * (D / 8); e += kMassThreads) {
    const int r = e / (D / 8), c = e - r * (D / 8);
    *(uint4*)(ks + r * ROW_BYTES + c * 16) = *(const uint4*)(kb + (int64_t)r * D + c * 8);
  }
  __syncthreads();

  const float c2 = a.sm_scale * 1.4426950408889634f;
  const int R = G * a.n_q;  // rows: head-major (hh * n_q + i)
  const int nn = lane & 31, gs = lane >> 5;
  const int n_kblk = (lbs + 31) / 32;
  const int n_rblk = (R + 31) / 32;
  // This lane's query pieces of row block rb (the B operand: row 32*rb + nn, dims
  // 16s + 8*gs .. +8; under the remap turned by R(l_L) and rounded to bf16, as the
  // attention does for memory keys) and the row's lse in the exp2 domain.
  auto load_rows = [&](int rb, bf16x8 (&qf)[KSTEPS], float& lse2, bool& ok) {
    const int row = rb * 32 + nn;
    ok = rb < n_rblk && row < R;
    const int hh = ok ? row / a.n_q : 0, qi = ok ? row - hh * a.n_q : 0;
    const int qh = g * G + hh;
    const bf16_t* qp = (const bf16_t*)a.q + (int64_t)(b * a.n_q_heads + qh) * a.q_head_stride + (int64_t)qi * D;
    u32x4 raw[KSTEPS];
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) raw[s] = ok ? *(const u32x4*)(qp + 16 * s + 8 * gs) : u32x4{0, 0, 0, 0};
    lse2 = ok ? a.lse[(int64_t)(b * a.n_q_heads + qh) * a.n_q + qi] * 1.4426950408889634f : __builtin_inff();
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      if (a.rope.on) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int pr = 8 * s + 4 * gs + j;
          const float cs = a.rope.mem_cos[pr], sn = a.rope.mem_sin[pr];
          const float x0 = __uint_as_float(raw[s][j] << 16), x1 = __uint_as_float(raw[s][j] & 0xFFFF0000u);
          raw[s][j] = (uint32_t)f32_to_bf16(x0 * cs - x1 * sn) | ((uint32_t)f32_to_bf16(x0 * sn + x1 * cs) << 16);
        }
      }
      qf[s] = __builtin_bit_cast(bf16x8, raw[s]);
    }
  };
  // p = exp2(S*c2 - lse2) over a 32x32 block (lane: row nn, keys 32*kbk + 8*(j/4)
  // + 4*gs + j%4).  A row past R carries lse2 = +inf (p = 0); keys past l_bs are
  // left out in the last, partial key block only.
  auto add_block = [&](const f32x16& sacc, int kbk, float lse2, float& acc) {
    if (32 * kbk + 32 <= lbs) {
#pragma unroll
      for (int j = 0; j < 16; ++j) acc += __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[j], c2, -lse2));
    } else {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int key = 32 * kbk + 8 * (j >> 2) + 4 * gs + (j & 3);
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[j], c2, -lse2));
        acc += key < lbs ? p : 0.f;
      }
    }
  };
  auto kfrag = [&](int kbk, int s) {
    const int kr = min(32 * kbk + nn, lbs - 1);  // clamped; masked in add_block
    return *(const bf16x8*)(ks + kr * ROW_BYTES + (16 * s + 8 * gs) * 2);
  };
  // Each wave takes two row blocks at a time: every K fragment read from LDS feeds
  // two independent accumulator chains, and the next fragment is read one k-step
  // ahead.
  float acc0 = 0.f, acc1 = 0.f;
  for (int rb = 2 * wave; rb < n_rblk; rb += 2 * kMassWaves) {
    bf16x8 qa[KSTEPS], qb[KSTEPS];
    float la, lb;
    bool oka, okb;
    load_rows(rb, qa, la, oka);
    load_rows(rb + 1, qb, lb, okb);
    for (int kbk = 0; kbk < n_kblk; ++kbk) {
      f32x16 sa = {}, sb = {};
      bf16x8 kf[2];
      kf[0] = kfrag(kbk, 0);
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
        if (s + 1 < KSTEPS) kf[(s + 1) & 1] = kfrag(kbk, s + 1);
        sa = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s & 1], qa[s], sa, 0, 0, 0);
        sb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s & 1], qb[s], sb, 0, 0, 0);
      }
      add_block(sa, kbk, la, acc0);
      add_block(sb, kbk, lb, acc1);
    }
  }
  const float acc = acc0 + acc1;
  const float tot = block_sum(acc, red);
  if (tid == 0) {
    a.mass[(int64_t)bg * a.k + slot] = tot;
    if (a.freq != nullptr) {
      float* f = a.freq + (int64_t)bg * a.max_units + unit;
      *f = *f * a.decay + tot;
    }
  }
}

// Mass of one looked-up unit, float32 inputs: one (row, key) pair per thread step.
template <int D>
__device__ void unit_mass_f32(const MassArgs& a, int bg, int slot, int unit, float* red) {
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int lbs = a.block_size;
  const float* kb = (const float*)a.k_store + ((int64_t)bg * a.capacity + a.n_init + (int64_t)unit * lbs) * D;
  const int R = G * a.n_q;
  float acc = 0.f;
  for (int e = threadIdx.x; e < R * lbs; e += kMassThreads) {
    const int row = e / lbs, key = e - row * lbs;
    const int hh = row / a.n_q, qi = row - hh * a.n_q;
    const int qh = g * G + hh;
    const float* qp = (const float*)a.q + (int64_t)(b * a.n_q_heads + qh) * a.q_head_stride + (int64_t)qi * D;
    const float* kp = kb + (int64_t)key * D;
    float z = 0.f;
    for (int d = 0; d < D; d += 2) {
      float x0 = qp[d], x1 = qp[d + 1];
      if (a.rope.on) {
        const float cs = a.rope.mem_cos[d / 2], sn = a.rope.mem_sin[d / 2];
        const float y0 = x0 * cs - x1 * sn, y1 = x0 * sn + x1 * cs;
        x0 = y0;
        x1 = y1;
      }
      z += x0 * kp[d] + x1 * kp[d + 1];
    }
    const float lse = a.lse[(int64_t)(b * a.n_q_heads + qh) * a.n_q + qi];
    acc += expf(a.sm_scale * z - lse);
  }
  const float tot = block_sum(acc, red);
  if (threadIdx.x == 0) {
    a.mass[(int64_t)bg * a.k + slot] = tot;
    if (a.freq != nullptr) {
      float* f = a.freq + (int64_t)bg * a.max_units + unit;
      *f = *f * a.decay + tot;
    }
  }
}

template <typename T, int D>
__global__ void __launch_bounds__(kMassThreads) mass_kernel(MassArgs a) {
  __shared__ float red[kMassWaves];
  __shared__ int sel[kMassMaxK];
  const int n_slot_blocks = a.rows * a.k;
  if ((int)blockIdx.x >= n_slot_blocks) {
    // decay of the scores of the units this row did not look up
    const int bg = blockIdx.x - n_slot_blocks;
    const int32_t* idx_row = a.idx + (int64_t)bg * a.k;
    for (int j = threadIdx.x; j < a.k; j += kMassThreads) sel[j] = idx_row[j];
    __syncthreads();
    float* f = a.freq + (int64_t)bg * a.max_units;
    for (int u = threadIdx.x; u < a.n_units; u += kMassThreads) {
      bool looked_up = false;
      for (int j = 0; j < a.k; ++j) looked_up |= sel[j] == u;
      if (!looked_up) f[u] *= a.decay;
    }
    return;
  }
  // the slots of one row go to one XCD, whose L2 then holds the row's queries
  const int L = xcd_logical_block(blockIdx.x, n_slot_blocks);
  const int bg = L / a.k, slot = L - bg * a.k;
  const int unit = a.idx[(int64_t)bg * a.k + slot];
  if (unit < 0 || unit >= a.n_units) {
    if (threadIdx.x == 0) a.mass[(int64_t)bg * a.k + slot] = 0.f;
    return;
  }
  if constexpr (sizeof(T) == 2) unit_mass_bf16<D>(a, bg, slot, unit, red);
  else unit_mass_f32<D>(a, bg, slot, unit, red);
}

// Unit masses from the attention's per-tile partials: one workgroup per (kv row,
// lookup slot) sums P_sum * exp2(m - lse2) over the unit's tiles and the rows in
// a fixed order; extra workgroups decay the units not looked up.
constexpr int kPartsThreads = 256;
constexpr int kPartsRows = 8;                              // rows per thread per load batch
constexpr int kMaxTilesPerUnit = kMassMaxBlock / 64;  // 64-key tiles of the longest unit
__global__ void __launch_bounds__(kPartsThreads) mass_parts_kernel(MassPartsArgs a) {
  __shared__ float red[kPartsThreads / 64];
  __shared__ int sel[kMassMaxK];
  const int n_slot_blocks = a.rows * a.k;
  if ((int)blockIdx.x >= n_slot_blocks) {
    const int bg = blockIdx.x - n_slot_blocks;
    decay_unselected<4>(a.idx + (int64_t)bg * a.k, a.k, a.freq + (int64_t)bg * a.max_units, a.n_units, a.decay, sel);
    return;
  }
  const int bg = blockIdx.x / a.k, slot = blockIdx.x - bg * a.k;
  if (slot >= a.n_sel) {
    if (threadIdx.x == 0) a.mass[(int64_t)bg * a.k + slot] = 0.f;
    return;
  }
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
  const int G = a.n_q_heads / a.n_kv_heads, R = G * a.n_q;
  const float* lse_g = a.lse + (int64_t)(b * a.n_q_heads + g * G) * a.n_q;  // head hh at lse_g + hh * n_q
  // Each thread takes kPartsRows rows per batch; all of a batch's loads (the rows'
  // lse and their partials in every tile of the unit) are issued before the first
  // use, so a batch costs one memory round trip.
  const float2* mp = a.mass_part + ((int64_t)bg * a.mass_tiles + (int64_t)slot * a.tiles_per_unit) * R;
  float acc = 0.f;
  // (indices past the row count or the unit's tiles are clamped, so that every
  // load is unconditional, and their terms dropped after)
  for (int base = 0; base < R; base += kPartsThreads * kPartsRows) {
    float lr[kPartsRows];
    float2 e[kMaxTilesPerUnit][kPartsRows];
#pragma unroll
    for (int j = 0; j < kPartsRows; ++j) {
      const int r = min(base + j * kPartsThreads + (int)threadIdx.x, R - 1);
      const int i = r / G, hh = r - i * G;  // attention rows are query-major
      lr[j] = lse_g[(int64_t)hh * a.n_q + i];
#pragma unroll
      for (int t = 0; t < kMaxTilesPerUnit; ++t) e[t][j] = mp[(int64_t)min(t, a.tiles_per_unit - 1) * R + r];
    }
#pragma unroll
    for (int t = 0; t < kMaxTilesPerUnit; ++t)
#pragma unroll
      for (int j = 0; j < kPartsRows; ++j) {
        const float term = e[t][j].x * __builtin_amdgcn_exp2f(e[t][j].y - lr[j] * 1.4426950408889634f);
        acc += (t < a.tiles_per_unit && base + j * kPartsThreads + (int)threadIdx.x < R) ? term : 0.f;
      }
  }
  const float tot = block_sum<kPartsThreads / 64>(acc, red);
  if (threadIdx.x == 0) {
    a.mass[(int64_t)bg * a.k + slot] = tot;
    if (a.freq != nullptr) {
      float* f = a.freq + (int64_t)bg * a.max_units + a.idx[(int64_t)bg * a.k + slot];
      *f = *f * a.decay + tot;
    }
  }
}

}  // namespace

hipError_t launch_unit_mass_parts(const MassPartsArgs& a, hipStream_t s) {
  const int blocks = a.rows * a.k + (a.freq != nullptr ? a.rows : 0);
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(mass_parts_kernel, dim3(blocks), dim3(kPartsThreads), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_unit_mass(const MassArgs& a, hipStream_t s) {
  const int blocks = a.rows * a.k + (a.freq != nullptr ? a.rows : 0);
  if (blocks == 0) return hipSuccess;
  const dim3 grid(blocks), block(kMassThreads);
  if (a.bf16) {
    if (a.head_dim == 128) hipLaunchKernelGGL((mass_kernel<bf16_t, 128>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((mass_kernel<bf16_t, 64>), grid, block, 0, s, a);
  } else {
    if (a.head_dim == 128) hipLaunchKernelGGL((mass_kernel<float, 128>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((mass_kernel<float, 64>), grid, block, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace infllm
