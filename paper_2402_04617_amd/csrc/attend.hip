// Attention dispatch (bfloat16 chunks: matrix-core kernel; bfloat16 decoding:
// the bandwidth kernel of attend_decode.hip), plus the float32 kernel:
//  - attend_f32_kernel: float32 inputs (any n_q), vector ALU, exact-exp online
//    softmax; the float32 accuracy path.  It reads keys through the same
//    virtual key axis as the other kernels; with the positional remap it holds
//    both forms of the query and picks one per key (memory or local).
#include "launch.h"

namespace infllm {

hipError_t launch_attend_mfma(const AttendArgs& a, hipStream_t s);
hipError_t launch_attend_decode(const AttendArgs& a, hipStream_t s);

namespace {

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

  const int G = a.n_q_heads / a.n_kv_heads;
  const int R = G * a.geom.n_q;
  const int n_row_tiles = (R + RW - 1) / RW;
  const int L = xcd_logical_block(blockIdx.x, gridDim.x);
  const int rt = L % n_row_tiles;
  const int tmp = L / n_row_tiles;
  const int part = tmp % a.parts;
  const int bg = tmp / a.parts;
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
  // this sequence's step (its own past length in a variable-length batch)
  const SeqStep sq = seq_step(a, b);
  const StepGeom& geo = sq.geom;
  const int mem_len = sq.mem_len, parts_mem = sq.parts_mem;

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

  // Query pieces: qv as given; with the positional remap qv is the query at its
  // own position (for L and X) and qm the query turned by R(l_L) (for I and the
  // units, whose keys are read unrotated).
  float qv[DPT], qm[DPT], o[DPT];
  const float* qp = (const float*)a.q + (int64_t)(b * a.n_q_heads + qh) * a.q_head_stride + (int64_t)qi * D;
#pragma unroll
  for (int e = 0; e < DPT; ++e) {
    qv[e] = row_ok ? qp[sub * DPT + e] : 0.f;
    qm[e] = qv[e];
    o[e] = 0.f;
  }
  const bool remap = a.rope.on != 0;
  const float* krot = (const float*)a.k_rot + (int64_t)bg * a.capacity * D;
  if (remap) {
#pragma unroll
    for (int j = 0; j < DPT / 2; ++j) {
      const int pr = sub * DPT / 2 + j;
      const float x0 = qv[2 * j], x1 = qv[2 * j + 1];
      float c, sn;
      rope_cos_sin(a.rope, geo.past_len + qi, pr, c, sn);
      qv[2 * j] = x0 * c - x1 * sn;
      qv[2 * j + 1] = x0 * sn + x1 * c;
      qm[2 * j] = x0 * a.rope.mem_cos[pr] - x1 * a.rope.mem_sin[pr];
      qm[2 * j + 1] = x0 * a.rope.mem_sin[pr] + x1 * a.rope.mem_cos[pr];
    }
  }
  float m = -__builtin_inff(), l = 0.f;

  for (int t = t_begin; t < t_end; ++t) {
    for (int e = tid; e < KT * D / 4; e += 256) {
      const int j = e / (D / 4), c = e - j * (D / 4);
      const int v = t * KT + j;
      const int64_t pos = v < geo.n_virtual ? virtual_pos(geo, idx_row, v) : -1;
      float4 kk = make_float4(0.f, 0.f, 0.f, 0.f), vv = kk;
      if (pos >= 0) {
        kk = *(const float4*)((remap && v >= mem_len ? krot : kbase) + pos * D + 4 * c);
        vv = *(const float4*)(vbase + pos * D + 4 * c);
      }
      *(float4*)&ks[j][4 * c] = kk;
      *(float4*)&vs[j][4 * c] = vv;
      if (c == 0) kval[j] = pos >= 0;
    }
    __syncthreads();
    for (int j = 0; j < KT; ++j) {
      const bool mem_key = remap && t * KT + j < mem_len;  // uniform over the workgroup
      float part_dot = 0.f;
#pragma unroll
      for (int e = 0; e < DPT; ++e) part_dot += (mem_key ? qm[e] : qv[e]) * ks[j][sub * DPT + e];
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
    float* op = (float*)a.part_o + ((int64_t)part * rows_total + grow) * D;
#pragma unroll
    for (int e = 0; e < DPT; ++e) op[sub * DPT + e] = o[e] * inv;
    if (sub == 0) a.part_lse[(int64_t)part * rows_total + grow] = lse_v;
  }
}

bool decode_eligible(bool bf16, int n_q, int G, int n_sel) {
  return bf16 && n_q == 1 && (G == 1 || G == 2 || G == 4 || G == 8) && n_sel <= kDecodeMaxSel;
}

}  // namespace

// Key parts of the decode kernel: enough workgroups for the whole chip, but at
// least kDecodeMinKeysPerWg keys each.
int attend_decode_parts(int bh, int n_virtual) {
  const int by_chip = (kDecodeTargetWgs + bh - 1) / bh;
  const int by_keys = max(1, n_virtual / kDecodeMinKeysPerWg);
  return max(1, min(by_chip, by_keys));
}

int attend_choose_parts(bool bf16, int batch, int n_q_heads, int n_kv_heads, int n_q, int n_sel, int n_virtual,
                        int max_parts) {
  const int G = n_q_heads / n_kv_heads;
  if (decode_eligible(bf16, n_q, G, n_sel)) return min(attend_decode_parts(batch * n_kv_heads, n_virtual), max(1, max_parts));
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
  if (decode_eligible(bf16, n_q, G, 0)) return attend_decode_parts(1, (int)max_virtual);
  return bf16 ? 8 : 16;
}

bool attend_uses_mfma(const AttendArgs& a) {
  const int G = a.n_q_heads / a.n_kv_heads;
  return a.geom.n_q > 0 && a.bf16 && !decode_eligible(a.bf16, a.geom.n_q, G, a.geom.n_sel);
}

hipError_t launch_attend(const AttendArgs& a, hipStream_t s) {
  if (a.geom.n_q == 0) return hipSuccess;
  const int G = a.n_q_heads / a.n_kv_heads;
  if (decode_eligible(a.bf16, a.geom.n_q, G, a.geom.n_sel)) return launch_attend_decode(a, s);
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
