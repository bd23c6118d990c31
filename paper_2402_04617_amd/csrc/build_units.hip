// Memory-unit construction (Section 3.2, "Block-Level Memory Units").
//
// One workgroup per (unit, sequence*kv head).  Each token m of the unit gets
// r_m = k_m . W_m with W_m = Pi_{m+l_L} - Pi_m read from the float64 running-sum
// ring (slot t holds the group's query sum through position t), which equals
// sum_{h in group} sum_{j=1..l_L} q^h_{m+j} . k_m.  The r_k tokens of largest r_m
// (ties: lower position) become R(B); the unit stores their offsets and the sum
// of their keys (what unit scoring streams).
#include "launch.h"

namespace infllm {
namespace {

constexpr int kMaxBlock = 256;

template <typename T>
__global__ void __launch_bounds__(256) build_units_kernel(BuildArgs a) {
  const int unit_local = blockIdx.x;
  const int unit = a.first_unit + unit_local;
  const int bg = blockIdx.y;
  const int D = a.head_dim;
  const int lbs = a.block_size;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t m0 = (int64_t)a.n_init + (int64_t)unit * lbs;
  const T* kb = (const T*)a.k_store + ((int64_t)bg * a.capacity) * D;
  const double* ring = a.qprefix + (int64_t)bg * a.ring * D;

  __shared__ double r[kMaxBlock];
  __shared__ int sel[kMaxBlock];
  __shared__ int chosen[kMaxBlock];

  // r_m for every token of the unit, one wave per token.
  for (int t = wave; t < lbs; t += 4) {
    const int64_t m = m0 + t;
    const double* hi = ring + ((m + a.n_local) % a.ring) * D;
    const double* lo = ring + (m % a.ring) * D;
    const T* km = kb + m * D;
    double acc = 0.0;
    for (int d = lane; d < D; d += 64) acc += (double)Elem<T>::load(km + d) * (hi[d] - lo[d]);
    acc = wave_sum_f64(acc);
    if (lane == 0) r[t] = (acc != acc) ? -__builtin_inf() : acc;  // NaN ranks lowest
  }
  __syncthreads();

  // Rank under the strict order (larger r first, then lower offset): exactly
  // the r_k tokens of rank < r_k are representatives.
  for (int t = threadIdx.x; t < lbs; t += blockDim.x) {
    const double rt = r[t];
    int rank = 0;
    for (int u = 0; u < lbs; ++u) {
      const double ru = r[u];
      rank += (ru > rt) || (ru == rt && u < t);
    }
    sel[t] = rank < a.n_repr;
  }
  __syncthreads();
  for (int t = threadIdx.x; t < lbs; t += blockDim.x) {
    if (sel[t]) {
      int slot = 0;
      for (int u = 0; u < t; ++u) slot += sel[u];
      chosen[slot] = t;
      a.repr_idx[((int64_t)bg * a.max_units + unit) * a.n_repr + slot] = t;
    }
  }
  __syncthreads();

  // Sum of the representative keys, in ascending position order, float32.
  for (int d = threadIdx.x; d < D; d += blockDim.x) {
    float s = 0.f;
    for (int j = 0; j < a.n_repr; ++j) s += Elem<T>::load(kb + (m0 + chosen[j]) * D + d);
    a.unit_ksum[(((int64_t)bg * (D / 4) + d / 4) * a.max_units + unit) * 4 + (d & 3)] = s;
  }
  if (a.repr_score != nullptr) {
    const int G = a.n_q_heads / a.n_kv_heads;
    const double norm = 1.0 / ((double)a.n_local * (double)G);
    for (int t = threadIdx.x; t < lbs; t += blockDim.x)
      a.repr_score[((int64_t)bg * a.n_new + unit_local) * lbs + t] = r[t] * norm;
  }
}

}  // namespace

hipError_t launch_build_units(const BuildArgs& a, hipStream_t s) {
  if (a.n_new == 0) return hipSuccess;
  dim3 grid(a.n_new, a.batch * a.n_kv_heads);
  if (a.bf16)
    hipLaunchKernelGGL(build_units_kernel<bf16_t>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(build_units_kernel<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace infllm
