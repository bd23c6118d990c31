// Unit relevance (Section 3.2, "memory lookup").
//
// sim(X, B) = sum_i sum_j q_{i+l_P} . k_{b_j} is bilinear, so per kv head it is
// Qbar . Kbar_B with Qbar the sum of the group's current queries and Kbar_B the
// sum of the unit's representative keys (kept by unit construction).  Qbar is the
// sum of the queries as given (unrotated when the positional remap is on).  Two
// kernels: a reduction of the chunk's queries into per-part partial sums
// (deterministic order), then one streaming pass over the Kbar table (fp32,
// unit-contiguous 16-byte cells) at HBM rate.
#include "qsum.h"

namespace infllm {
namespace {

constexpr int kMaxQbarParts = 16;

// grid (parts, batch*Hkv)
template <typename T>
__global__ void __launch_bounds__(kQsumThreads) qbar_kernel(const T* __restrict__ q, int64_t q_head_stride,
                                                            int n_q_heads, int n_kv_heads, int head_dim,
                                                            int n_q, int parts, float* __restrict__ qbar_parts) {
  __shared__ QsumSmem<T> sm;
  qsum_block<T>(q, q_head_stride, n_q_heads, n_kv_heads, head_dim, n_q, blockIdx.x, parts, blockIdx.y, qbar_parts,
                sm);
}

// grid (ceil(n_units/64), batch*Hkv); 64 units per block, each unit's D dims
// split over the block's 4 waves (wave w takes 16-byte cells [w*D/16, (w+1)*D/16)),
// so that a wave's load of one cell covers 64 consecutive units (1 KB) and a
// chunk's few hundred units still spread over many compute units.  Every thread
// issues its D/16 loads first, so that they are in flight while the block forms
// Qbar (the sum of the query-sum partials, turned by R(l_L) under the positional
// remap: the memory keys sit at distance l_L from every current token and stay
// unrotated); the four partial dot products of a unit are added in LDS in a
// fixed order.  In a variable-length batch sequence b scores its own unit count
// (units past it are left alone) into rows of stride score_stride.
constexpr int kScoreUnits = 64;
template <int D>
__global__ void __launch_bounds__(256) score_kernel(const ScoreArgs a, int parts) {
  constexpr int NC = D / 4;   // 16-byte cells per unit
  constexpr int CPW = NC / 4;  // cells per wave
  const int bg = blockIdx.y;
  const int n_units = a.var_on ? a.var_units[bg / a.n_kv_heads] : a.n_units;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int u = blockIdx.x * kScoreUnits + lane;
  const bool live = u < n_units;
  // a thread past the last unit reads unit 0 (always present) and stores nothing
  const float4* ks = (const float4*)a.unit_ksum + (int64_t)bg * NC * a.max_units + (live ? u : 0);
  float4 k4[CPW];
#pragma unroll
  for (int c = 0; c < CPW; ++c) k4[c] = ks[(int64_t)(w * CPW + c) * a.max_units];

  const RopeArgs& rope = a.rope;
  __shared__ float qbar[D];
  __shared__ float part[4][kScoreUnits];
  if (threadIdx.x < D) {
    // every part's load issued before the first add (a loop that waits for each
    // load in turn would also wait behind the key-sum loads above)
    const float* qp = a.qbar_parts + (int64_t)bg * parts * D + threadIdx.x;
    float s = 0.f;
    if (parts == 1) {
      s = *qp;
    } else {
      float v[kMaxQbarParts];
#pragma unroll
      for (int p = 0; p < kMaxQbarParts; ++p) v[p] = p < parts ? qp[p * D] : 0.f;
#pragma unroll
      for (int p = 0; p < kMaxQbarParts; ++p)
        if (p < parts) s += v[p];
    }
    qbar[threadIdx.x] = s;
  }
  __syncthreads();
  if (rope.on) {
    const int i = threadIdx.x;
    float x0 = 0.f, x1 = 0.f, c = 1.f, sn = 0.f;
    if (i < D / 2) {
      x0 = qbar[2 * i];
      x1 = qbar[2 * i + 1];
      c = rope.mem_cos[i];
      sn = rope.mem_sin[i];
    }
    __syncthreads();
    if (i < D / 2) {
      qbar[2 * i] = x0 * c - x1 * sn;
      qbar[2 * i + 1] = x0 * sn + x1 * c;
    }
    __syncthreads();
  }
  float acc = 0.f;
#pragma unroll
  for (int c = 0; c < CPW; ++c) {
    const int d = 4 * (w * CPW + c);
    acc += qbar[d] * k4[c].x + qbar[d + 1] * k4[c].y + qbar[d + 2] * k4[c].z + qbar[d + 3] * k4[c].w;
  }
  part[w][lane] = acc;
  __syncthreads();
  if (w == 0 && live)
    a.scores[(int64_t)bg * (a.var_on ? a.score_stride : n_units) + u] =
        ((part[0][lane] + part[1][lane]) + part[2][lane]) + part[3][lane];
}

}  // namespace

int score_qbar_parts(int G, int n_q) {
  int rows = G * n_q;
  int parts = (rows + 127) / 128;  // 128 rows per block: one batch of loads per thread
  return parts < 1 ? 1 : (parts > kMaxQbarParts ? kMaxQbarParts : parts);
}

hipError_t launch_score(const ScoreArgs& a, hipStream_t s) {
  if (a.n_units == 0) return hipSuccess;
  const int G = a.n_q_heads / a.n_kv_heads;
  const int parts = score_qbar_parts(G, a.n_q);
  dim3 g1(parts, a.batch * a.n_kv_heads);
  if (a.bf16)
    hipLaunchKernelGGL(qbar_kernel<bf16_t>, g1, dim3(kQsumThreads), 0, s, (const bf16_t*)a.q, a.q_head_stride,
                       a.n_q_heads, a.n_kv_heads, a.head_dim, a.n_q, parts, a.qbar_parts);
  else
    hipLaunchKernelGGL(qbar_kernel<float>, g1, dim3(kQsumThreads), 0, s, (const float*)a.q, a.q_head_stride,
                       a.n_q_heads, a.n_kv_heads, a.head_dim, a.n_q, parts, a.qbar_parts);
  return launch_score_given_qbar(a, parts, s);
}

hipError_t launch_score_given_qbar(const ScoreArgs& a, int parts, hipStream_t s) {
  if (a.n_units == 0) return hipSuccess;
  dim3 g2((a.n_units + kScoreUnits - 1) / kScoreUnits, a.batch * a.n_kv_heads);  // n_units: the largest of the batch
  if (a.head_dim == 128) hipLaunchKernelGGL(score_kernel<128>, g2, dim3(256), 0, s, a, parts);
  else hipLaunchKernelGGL(score_kernel<64>, g2, dim3(256), 0, s, a, parts);
  return hipGetLastError();
}

}  // namespace infllm
