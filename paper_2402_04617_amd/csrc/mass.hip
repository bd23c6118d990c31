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
// One workgroup per (sequence*kv head, lookup slot).  bf16: the unit's keys are
// staged in LDS once (rows padded by 16 bytes so the fragment reads of 32 rows
// spread over the banks), each wave takes 32-row blocks of the group's queries
// as the B operand of v_mfma_f32_32x32x16_bf16 against 32-key blocks of the
// unit, exponentiates against the row's lse and accumulates; one float per lane,
// then a wave and a workgroup sum.  float32: plain dot products per (row, key).
// Extra workgroups, one per (sequence*kv head), decay the scores of the units
// not looked up, so every score is written by exactly one thread.
#include "launch.h"

namespace infllm {
namespace {

constexpr int kMassThreads = 512;
constexpr int kMassWaves = kMassThreads / 64;
constexpr int kMassMaxBlock = 256;  // largest l_bs

// Sum of a float over the workgroup (every thread gets it).
__device__ __forceinline__ float block_sum(float x, float* red) {
  x = wave_sum(x);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) red[wave] = x;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int w = 0; w < kMassWaves; ++w) t += red[w];
  return t;
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
  float acc = 0.f;
  const int nn = lane & 31, gs = lane >> 5;
  const int n_kblk = (lbs + 31) / 32;
  for (int rb = wave; rb * 32 < R; rb += kMassWaves) {
    const int row = rb * 32 + nn;
    const bool row_ok = row < R;
    const int hh = row_ok ? row / a.n_q : 0, qi = row_ok ? row - hh * a.n_q : 0;
    const int qh = g * G + hh;
    // this lane's query pieces (B operand): row `row`, dims 16s + 8*gs .. +8
    const bf16_t* qp = (const bf16_t*)a.q + (int64_t)(b * a.n_q_heads + qh) * a.q_head_stride + (int64_t)qi * D;
    bf16x8 qf[KSTEPS];
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      u32x4 raw = row_ok ? *(const u32x4*)(qp + 16 * s + 8 * gs) : u32x4{0, 0, 0, 0};
      if (a.rope.on) {
        // memory keys meet the query turned by R(l_L), rounded to bf16 as the attention does
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int pr = 8 * s + 4 * gs + j;
          const float cs = a.rope.mem_cos[pr], sn = a.rope.mem_sin[pr];
          const float x0 = __uint_as_float(raw[j] << 16), x1 = __uint_as_float(raw[j] & 0xFFFF0000u);
          raw[j] = (uint32_t)f32_to_bf16(x0 * cs - x1 * sn) | ((uint32_t)f32_to_bf16(x0 * sn + x1 * cs) << 16);
        }
      }
      qf[s] = __builtin_bit_cast(bf16x8, raw);
    }
    const float lse2 = row_ok ? a.lse[(int64_t)(b * a.n_q_heads + qh) * a.n_q + qi] * 1.4426950408889634f : 0.f;
    for (int kbk = 0; kbk < n_kblk; ++kbk) {
      f32x16 sacc = {};
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
        // A operand: key row 32*kbk + nn (clamped; masked below), dims 16s + 8*gs
        const int kr = min(32 * kbk + nn, lbs - 1);
        const bf16x8 kf = *(const bf16x8*)(ks + kr * ROW_BYTES + (16 * s + 8 * gs) * 2);
        sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s], sacc, 0, 0, 0);
      }
      // lane holds column nn (this row) and keys 8*(j/4) + 4*gs + j%4 of the block
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int key = 32 * kbk + 8 * (j >> 2) + 4 * gs + (j & 3);
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[j], c2, -lse2));
        acc += (row_ok && key < lbs) ? p : 0.f;
      }
    }
  }
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

}  // namespace

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
