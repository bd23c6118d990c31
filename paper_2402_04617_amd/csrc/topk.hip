// Top-k unit lookup (Section 3.2: only the k_m units of highest relevance are loaded).
//
// One workgroup per row running the radix select of topk_select.h.
#include "topk_select.h"

namespace infllm {
namespace {

using tk::kThreads;
using tk::kWaves;
using tk::kMaxPer;

// PER: keys per thread of the common path (0: radix select only).
// Rows of a variable-length batch (var_on): row r holds tr.row_n[r / rows_per_seq]
// scores; n is then the largest of them.  Rows are `stride` floats apart.
template <int PER>
__global__ void __launch_bounds__(kThreads) topk_kernel(const float* __restrict__ scores, int stride, int n_all,
                                                        int k, int32_t* __restrict__ idx, const TopkRows tr,
                                                        int var_on) {
  const int row = blockIdx.x;
  const int n = var_on ? tr.row_n[row / tr.rows_per_seq] : n_all;
  const float* s = scores + (int64_t)row * stride;
  int32_t* out = idx + (int64_t)row * k;
  const int k_eff = min(k, n);
  for (int j = k_eff + threadIdx.x; j < k; j += kThreads) out[j] = -1;
  if (k_eff == 0) return;
  __shared__ int wave_tot[kWaves];
  if constexpr (PER > 0) {
    if (k_eff < n) {
      tk::radix_select_reg<PER>(s, n, k_eff, out);
      return;
    }
  }
  tk::radix_select(s, n, k_eff, out, wave_tot);
}

}  // namespace

static hipError_t launch_topk(int rows, const float* scores, int stride, int n_max, const TopkRows& tr, int var_on,
                              int k, int32_t* idx, hipStream_t s) {
  if (rows == 0 || k == 0) return hipSuccess;
  const int per = (n_max + kThreads - 1) / kThreads;
  const dim3 grid(rows), block(kThreads);
#define INFLLM_TOPK(P) hipLaunchKernelGGL(topk_kernel<P>, grid, block, 0, s, scores, stride, n_max, k, idx, tr, var_on)
  if (per <= 1) INFLLM_TOPK(1);
  else if (per <= 2) INFLLM_TOPK(2);
  else if (per <= 4) INFLLM_TOPK(4);
  else if (per <= 8) INFLLM_TOPK(8);
  else if (per <= kMaxPer) INFLLM_TOPK(kMaxPer);
  else INFLLM_TOPK(0);
#undef INFLLM_TOPK
  return hipGetLastError();
}

hipError_t launch_select_topk(int rows, const float* scores, int n_units, int k, int32_t* idx,
                              hipStream_t s) {
  TopkRows tr;
  tr.rows_per_seq = 1;
  return launch_topk(rows, scores, n_units, n_units, tr, 0, k, idx, s);
}

hipError_t launch_select_topk_var(int rows, const float* scores, int stride, int n_max, const TopkRows& tr, int k,
                                  int32_t* idx, hipStream_t s) {
  return launch_topk(rows, scores, stride, n_max, tr, 1, k, idx, s);
}

}  // namespace infllm
