// Standalone unit-construction kernel (the routine itself is in unit_build.h).
#include "unit_build.h"

namespace infllm {
namespace {

template <typename T, int D>
__global__ void __launch_bounds__(1024) build_units_kernel(BuildArgs a) {
  __shared__ BuildSmem sm;
  construct_unit<T, D, 1024>(a, blockIdx.x, blockIdx.y, sm);
}

}  // namespace

hipError_t launch_build_units(const BuildArgs& a, hipStream_t s) {
  if (a.n_new == 0) return hipSuccess;
  dim3 grid(a.n_new, a.batch * a.n_kv_heads);
  if (a.bf16) {
    if (a.head_dim == 128) hipLaunchKernelGGL((build_units_kernel<bf16_t, 128>), grid, dim3(1024), 0, s, a);
    else hipLaunchKernelGGL((build_units_kernel<bf16_t, 64>), grid, dim3(1024), 0, s, a);
  } else {
    if (a.head_dim == 128) hipLaunchKernelGGL((build_units_kernel<float, 128>), grid, dim3(1024), 0, s, a);
    else hipLaunchKernelGGL((build_units_kernel<float, 64>), grid, dim3(1024), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace infllm
