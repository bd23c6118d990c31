// Attention dispatch, plus the two non-MFMA attention kernels:
//  - attend_f32_kernel: float32 inputs (any n_q), vector ALU, exact-exp online
//    softmax; the float32 accuracy path.
//  - attend_decode_kernel: bfloat16, one current token per sequence (l_X = 1,
//    decoding).  With only G query rows per kv head the step is bound by
//    streaming K/V from HBM, so each workgroup takes 256 keys of one
//    (sequence, kv head), scores them, and writes a partial softmax for the
//    log-sum-exp merge.
// Both read keys through the same virtual key axis as the MFMA kernel.
#include "launch.h"

namespace infllm {

hipError_t launch_attend_mfma(const AttendArgs& a, hipStream_t s);

namespace {

constexpr int kDecodeKeys = 256;

__device__ __forceinline__ bool key_visible(const StepGeom& geo, int v, int qi) {
  const int v_x0 = geo.n_virtual - geo.n_q;
  return v < geo.n_virtual && (v < v_x0 || v - v_x0 <= qi);
}

// ---------------------------------------------------------------- float32 path
template <int D>
__global__ void __launch_bounds__(256) attend_f32_kernel(AttendArgs a) {
  constexpr int RW = 16, TPR = 16, DPT = D / TPR, KT = 32;
  __shared__ __attribute__((aligned(16))) float ks[KT][D];
  __shared__ __attribute__((aligned(16))) float vs[KT][D];
  __shared__ int kval[KT];

  const StepGeom& geo = a.geom;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int R = G * geo.n_q;
  const int n_row_tiles = (R + RW - 1) / RW;
  const int L = xcd_logical_block(blockIdx.x, gridDim.x);
  const int rt = L % n_row_tiles;
  const int tmp = L / n_row_tiles;
  const int part = tmp % a.parts;
  const int bg = tmp / a.parts;
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;

  const int n_tiles = (geo.n_virtual + KT - 1) / KT;
  const int per_part = (n_tiles + a.parts - 1) / a.parts;
  const int t_begin = part * per_part;
  int t_end = min(n_tiles, t_begin + per_part);
  {
    const int i_max = (min(R, (rt + 1) * RW) - 1) / G;
    t_end = min(t_end, (geo.n_virtual - geo.n_q + i_max) / KT + 1);
  }

  const int tid = threadIdx.x;
  const int rl = tid / TPR, sub = tid % TPR;
  const int row = rt * RW + rl;
  const bool row_ok = row < R;
  const int qi = row_ok ? row / G : 0;
  const int qh = g * G + (row_ok ? row - qi * G : 0);
  const int32_t* idx_row = a.idx + (int64_t)bg * geo.idx_stride;
  const float* kbase = (const float*)a.k_store + (int64_t)bg * a.capacity * D;
  const float* vbase = (const float*)a.v_store + (int64_t)bg * a.capacity * D;

  float qv[DPT], o[DPT];
  const float* qp = (const float*)a.q + (int64_t)(b * a.n_q_heads + qh) * a.q_head_stride + (int64_t)qi * D;
#pragma unroll
  for (int e = 0; e < DPT; ++e) {
    qv[e] = row_ok ? qp[sub * DPT + e] : 0.f;
    o[e] = 0.f;
  }
  float m = -__builtin_inff(), l = 0.f;

  for (int t = t_begin; t < t_end; ++t) {
    for (int e = tid; e < KT * D / 4; e += 256) {
      const int j = e / (D / 4), c = e - j * (D / 4);
      const int v = t * KT + j;
      const int64_t pos = v < geo.n_virtual ? virtual_pos(geo, idx_row, v) : -1;
      float4 kk = make_float4(0.f, 0.f, 0.f, 0.f), vv = kk;
      if (pos >= 0) {
        kk = *(const float4*)(kbase + pos * D + 4 * c);
        vv = *(const float4*)(vbase + pos * D + 4 * c);
      }
      *(float4*)&ks[j][4 * c] = kk;
      *(float4*)&vs[j][4 * c] = vv;
      if (c == 0) kval[j] = pos >= 0;
    }
    __syncthreads();
    for (int j = 0; j < KT; ++j) {
      float part_dot = 0.f;
#pragma unroll
      for (int e = 0; e < DPT; ++e) part_dot += qv[e] * ks[j][sub * DPT + e];
#pragma unroll
      for (int off = TPR / 2; off > 0; off >>= 1) part_dot += __shfl_xor(part_dot, off);
      const bool vis = kval[j] && key_visible(geo, t * KT + j, qi);
      if (vis) {
        const float s = part_dot * a.sm_scale;
        const float m_new = fmaxf(m, s);
        const float corr = expf(m - m_new);
        const float p = expf(s - m_new);
        l = l * corr + p;
#pragma unroll
        for (int e = 0; e < DPT; ++e) o[e] = o[e] * corr + p * vs[j][sub * DPT + e];
        m = m_new;
      }
    }
    __syncthreads();
  }

  if (!row_ok) return;
  const float inv = l > 0.f ? 1.f / l : 0.f;
  const float lse_v = l > 0.f ? m + logf(l) : -__builtin_inff();
  const int64_t grow = (int64_t)(b * a.n_q_heads + qh) * geo.n_q + qi;
  if (a.parts == 1) {
    float* op = (float*)a.out + (int64_t)(b * a.n_q_heads + qh) * a.out_head_stride + (int64_t)qi * D;
#pragma unroll
    for (int e = 0; e < DPT; ++e) op[sub * DPT + e] = o[e] * inv;
    if (a.lse != nullptr && sub == 0) a.lse[grow] = lse_v;
  } else {
    const int64_t rows_total = (int64_t)a.batch * a.n_q_heads * geo.n_q;
    float* op = a.part_o + ((int64_t)part * rows_total + grow) * D;
#pragma unroll
    for (int e = 0; e < DPT; ++e) op[sub * DPT + e] = o[e] * inv;
    if (sub == 0) a.part_lse[(int64_t)part * rows_total + grow] = lse_v;
  }
}

// ---------------------------------------------------------------- bf16 decode
template <int D, int G>
__global__ void __launch_bounds__(256) attend_decode_kernel(AttendArgs a) {
  constexpr int CH = D / 8;            // 16-byte chunks per row
  constexpr int KG = 256 / CH;         // key groups in the value pass
  constexpr int QD = D / 4;            // dims per thread in the score pass
  __shared__ float q_s[G][D];
  __shared__ float sc[G][kDecodeKeys];
  __shared__ float red[KG][G][D];
  __shared__ float m_s[G], l_s[G];

  const StepGeom& geo = a.geom;
  const int part = blockIdx.x % a.parts;
  const int bg = blockIdx.x / a.parts;
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
  const int v0 = part * kDecodeKeys;
  const int nk = max(0, min(kDecodeKeys, geo.n_virtual - v0));
  const int tid = threadIdx.x;
  const int32_t* idx_row = a.idx + (int64_t)bg * geo.idx_stride;
  const bf16_t* kbase = (const bf16_t*)a.k_store + (int64_t)bg * a.capacity * D;
  const bf16_t* vbase = (const bf16_t*)a.v_store + (int64_t)bg * a.capacity * D;
  const float c2 = a.sm_scale * 1.4426950408889634f;

  for (int e = tid; e < G * D; e += 256) {
    const int h = e / D, d = e - h * D;
    q_s[h][d] = bf16_to_f32(((const bf16_t*)a.q)[(int64_t)(b * a.n_q_heads + g * G + h) * a.q_head_stride + d]);
  }
  __syncthreads();

  // Scores: 4 threads per key, each a quarter of the head dim.
  {
    const int kk = tid >> 2, dq = tid & 3;
    for (int pass = 0; pass < kDecodeKeys / 64; ++pass) {
      const int j = pass * 64 + kk;
      const int v = v0 + j;
      const int64_t pos = (j < nk) ? virtual_pos(geo, idx_row, v) : -1;
      float acc[G];
#pragma unroll
      for (int h = 0; h < G; ++h) acc[h] = 0.f;
      if (pos >= 0) {
        const bf16_t* kr = kbase + pos * D + dq * QD;
#pragma unroll
        for (int c = 0; c < QD / 8; ++c) {
          const uint4 raw = *(const uint4*)(kr + 8 * c);
          const bf16_t* kv = (const bf16_t*)&raw;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float kf = bf16_to_f32(kv[e]);
#pragma unroll
            for (int h = 0; h < G; ++h) acc[h] += kf * q_s[h][dq * QD + 8 * c + e];
          }
        }
      }
#pragma unroll
      for (int h = 0; h < G; ++h) {
        float x = acc[h];
        x += __shfl_xor(x, 1);
        x += __shfl_xor(x, 2);
        if (dq == 0) sc[h][j] = (pos >= 0) ? x * c2 : -__builtin_inff();
      }
    }
  }
  __syncthreads();

  // Softmax statistics per head (one wave per head, exp2 domain).
  {
    const int lane = tid & 63, wave = tid >> 6;
    for (int h = wave; h < G; h += 4) {
      float mx = -__builtin_inff();
      for (int j = lane; j < kDecodeKeys; j += 64) mx = fmaxf(mx, sc[h][j]);
      mx = wave_max(mx);
      const float base = (mx == -__builtin_inff()) ? 0.f : mx;
      float sum = 0.f;
      for (int j = lane; j < kDecodeKeys; j += 64) {
        const float p = __builtin_amdgcn_exp2f(sc[h][j] - base);
        sc[h][j] = p;
        sum += p;
      }
      sum = wave_sum(sum);
      if (lane == 0) {
        m_s[h] = mx;
        l_s[h] = sum;
      }
    }
  }
  __syncthreads();

  // Values: 16-byte chunks, key groups strided over the part.
  {
    const int kg = tid / CH, c = tid % CH;
    float acc[G][8];
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
    for (int j = kg; j < nk; j += KG) {
      const int64_t pos = virtual_pos(geo, idx_row, v0 + j);
      if (pos < 0) continue;
      const uint4 raw = *(const uint4*)(vbase + pos * D + 8 * c);
      const bf16_t* vv = (const bf16_t*)&raw;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float vf = bf16_to_f32(vv[e]);
#pragma unroll
        for (int h = 0; h < G; ++h) acc[h][e] += sc[h][j] * vf;
      }
    }
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) red[kg][h][8 * c + e] = acc[h][e];
  }
  __syncthreads();

  const int64_t rows_total = (int64_t)a.batch * a.n_q_heads;  // n_q == 1
  for (int e = tid; e < G * D; e += 256) {
    const int h = e / D, d = e - h * D;
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < KG; ++k) s += red[k][h][d];
    const float l = l_s[h];
    const float o = l > 0.f ? s / l : 0.f;
    const int64_t grow = (int64_t)b * a.n_q_heads + g * G + h;
    if (a.parts == 1) {
      ((bf16_t*)a.out)[(int64_t)(b * a.n_q_heads + g * G + h) * a.out_head_stride + d] = f32_to_bf16(o);
    } else {
      a.part_o[((int64_t)part * rows_total + grow) * D + d] = o;
    }
    if (d == 0) {
      const float lse_v = (l > 0.f) ? (m_s[h] + __log2f(l)) * 0.6931471805599453f : -__builtin_inff();
      if (a.parts == 1) {
        if (a.lse != nullptr) a.lse[grow] = lse_v;
      } else {
        a.part_lse[(int64_t)part * rows_total + grow] = lse_v;
      }
    }
  }
}

bool decode_eligible(bool bf16, int n_q, int G) { return bf16 && n_q == 1 && (G == 1 || G == 2 || G == 4 || G == 8); }

template <int D>
hipError_t launch_decode(const AttendArgs& a, hipStream_t s) {
  const int G = a.n_q_heads / a.n_kv_heads;
  dim3 grid(a.parts * a.batch * a.n_kv_heads);
  switch (G) {
    case 1: hipLaunchKernelGGL((attend_decode_kernel<D, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((attend_decode_kernel<D, 2>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((attend_decode_kernel<D, 4>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((attend_decode_kernel<D, 8>), grid, dim3(256), 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace

int attend_decode_parts(int n_virtual) { return (n_virtual + kDecodeKeys - 1) / kDecodeKeys; }

int attend_choose_parts(bool bf16, int batch, int n_q_heads, int n_kv_heads, int n_q, int n_virtual,
                        int max_parts) {
  const int G = n_q_heads / n_kv_heads;
  if (decode_eligible(bf16, n_q, G)) {
    const int p = attend_decode_parts(n_virtual);
    return p <= max(1, max_parts) ? p : -1;  // decode parts are fixed by the key count
  }
  const int rows_per_wg = bf16 ? kMfmaRowsPerWg : 16;
  const int key_tile = bf16 ? 64 : 32;
  const int cap = bf16 ? 8 : 16;
  const int target = bf16 ? kMfmaTargetWgs : 512;
  const int row_tiles = batch * n_kv_heads * ((G * n_q + rows_per_wg - 1) / rows_per_wg);
  const int n_tiles = (n_virtual + key_tile - 1) / key_tile;
  int p = (target + row_tiles - 1) / row_tiles;
  p = min(p, cap);
  p = min(p, max(1, n_tiles / 2));
  p = min(p, max(1, max_parts));
  return max(1, p);
}

int attend_max_parts(bool bf16, int G, int n_q, int64_t max_virtual) {
  if (decode_eligible(bf16, n_q, G)) return attend_decode_parts((int)max_virtual);
  return bf16 ? 8 : 16;
}

hipError_t launch_attend(const AttendArgs& a, hipStream_t s) {
  if (a.geom.n_q == 0) return hipSuccess;
  const int G = a.n_q_heads / a.n_kv_heads;
  if (decode_eligible(a.bf16, a.geom.n_q, G))
    return a.head_dim == 128 ? launch_decode<128>(a, s) : launch_decode<64>(a, s);
  if (a.bf16) return launch_attend_mfma(a, s);
  const int R = G * a.geom.n_q;
  const int blocks = ((R + 15) / 16) * a.parts * a.batch * a.n_kv_heads;
  if (a.head_dim == 128)
    hipLaunchKernelGGL(attend_f32_kernel<128>, dim3(blocks), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(attend_f32_kernel<64>, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace infllm
