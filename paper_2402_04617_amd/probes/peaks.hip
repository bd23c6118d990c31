// Measured peaks of the MI355X this runs on, for roofline fractions next to the
// published ones: a register-only bf16 MFMA loop (v_mfma_f32_32x32x16_bf16, four
// independent accumulator chains per wave, two waves per SIMD), a streaming HBM
// read (4 GiB, 16-byte loads, eight in flight per thread) and a streaming copy
// (1 GiB to 1 GiB, best of three grid sizes).  Prints one JSON line; exit
// status 1 on any HIP error.
#include <hip/hip_runtime.h>

#include <cstdio>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int kChains = 4;
constexpr int kIters = 4000;

__global__ void __launch_bounds__(256) mfma_loop(float* out, float seed) {
  bf16x8 a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(seed * (float)(threadIdx.x + i));
    b[i] = (__bf16)(seed * (float)(i + 1));
  }
  f32x16 c[kChains];
  for (int k = 0; k < kChains; ++k) c[k] = f32x16{};
  for (int it = 0; it < kIters / 4; ++it) {  // 16 MFMAs per loop trip
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int k = 0; k < kChains; ++k) c[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[k], 0, 0, 0);
  }
  float s = 0.f;
  for (int k = 0; k < kChains; ++k)
    for (int i = 0; i < 16; ++i) s += c[k][i];
  out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

constexpr int kUnroll = 8;

__global__ void __launch_bounds__(256) stream_read(const uint4* __restrict__ p, size_t n, uint32_t* out) {
  size_t i = (size_t)blockIdx.x * 256 * kUnroll + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * 256 * kUnroll;
  uint32_t acc = 0;
  for (; i + (kUnroll - 1) * 256 < n; i += stride) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = p[i + u * 256];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  out[(size_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

__global__ void __launch_bounds__(256) stream_copy(const uint4* __restrict__ src, uint4* __restrict__ dst, size_t n) {
  size_t i = (size_t)blockIdx.x * 256 * kUnroll + threadIdx.x;
  const size_t stride = (size_t)gridDim.x * 256 * kUnroll;
  for (; i + (kUnroll - 1) * 256 < n; i += stride) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) v[u] = src[i + u * 256];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) dst[i + u * 256] = v[u];
  }
}

bool ok(hipError_t e) { return e == hipSuccess; }

// Best of `reps` timed launches (after two warm-ups), in milliseconds; < 0 on error.
template <typename F>
float best_ms(F launch, int reps) {
  hipEvent_t a, b;
  if (!ok(hipEventCreate(&a)) || !ok(hipEventCreate(&b))) return -1.f;
  for (int w = 0; w < 2; ++w) launch();
  float best = 1e30f;
  for (int r = 0; r < reps; ++r) {
    if (!ok(hipEventRecord(a))) return -1.f;
    launch();
    if (!ok(hipEventRecord(b)) || !ok(hipEventSynchronize(b))) return -1.f;
    float ms = 0.f;
    if (!ok(hipEventElapsedTime(&ms, a, b))) return -1.f;
    best = ms < best ? ms : best;
  }
  if (!ok(hipGetLastError())) return -1.f;
  return best;
}

}  // namespace

int main() {
  const int mfma_blocks = 512;                // 256 compute units x two 4-wave workgroups
  const size_t read_bytes = (size_t)4 << 30;  // well beyond the 256 MB last-level cache
  const size_t copy_bytes = (size_t)1 << 30;
  const int stream_blocks = 1024;
  float* out = nullptr;
  uint4 *big = nullptr, *src = nullptr, *dst = nullptr;
  uint32_t* sink = nullptr;
  if (!ok(hipMalloc(&out, (size_t)mfma_blocks * 256 * sizeof(float))) || !ok(hipMalloc(&big, read_bytes)) ||
      !ok(hipMalloc(&src, copy_bytes)) || !ok(hipMalloc(&dst, copy_bytes)) ||
      !ok(hipMalloc(&sink, (size_t)stream_blocks * 256 * sizeof(uint32_t))) ||
      !ok(hipMemset(big, 1, read_bytes)) || !ok(hipMemset(src, 2, copy_bytes)) || !ok(hipDeviceSynchronize())) {
    fprintf(stderr, "peaks: allocation failed\n");
    return 1;
  }
  const float t_mfma = best_ms([&] { hipLaunchKernelGGL(mfma_loop, dim3(mfma_blocks), dim3(256), 0, 0, out, 1e-3f); }, 5);
  const float t_read = best_ms(
      [&] { hipLaunchKernelGGL(stream_read, dim3(stream_blocks), dim3(256), 0, 0, big, read_bytes / 16, sink); }, 5);
  float t_copy = 1e30f;
  const int one_pass = (int)(copy_bytes / 16 / (256 * kUnroll));  // every thread moves kUnroll vectors once
  for (int blocks : {stream_blocks, 4 * stream_blocks, one_pass}) {  // best of three grid sizes
    const float t = best_ms(
        [&] { hipLaunchKernelGGL(stream_copy, dim3(blocks), dim3(256), 0, 0, src, dst, copy_bytes / 16); }, 5);
    if (t <= 0.f) {
      t_copy = -1.f;
      break;
    }
    t_copy = t < t_copy ? t : t_copy;
  }
  if (t_mfma <= 0.f || t_read <= 0.f || t_copy <= 0.f) {
    fprintf(stderr, "peaks: a timed launch failed\n");
    return 1;
  }
  const double mfma_flops = (double)mfma_blocks * 4 * kIters * kChains * 32768.0;  // 4 waves per block
  printf("{\"mfma_bf16_tflops\": %.1f, \"hbm_read_gbs\": %.1f, \"hbm_copy_gbs\": %.1f}\n",
         mfma_flops / (t_mfma * 1e-3) / 1e12, (double)read_bytes / (t_read * 1e-3) / 1e9,
         2.0 * (double)copy_bytes / (t_copy * 1e-3) / 1e9);
  (void)hipFree(out);
  (void)hipFree(big);
  (void)hipFree(src);
  (void)hipFree(dst);
  (void)hipFree(sink);
  return 0;
}
