// The unit lookup's top-k (Section 3.2: the k_m units of highest relevance) two
// ways on the same score rows: a textbook bitonic top-k (each row's (score,
// index) keys fully sorted in LDS by a bitonic network, the first k kept) and
// the library's radix select (infllm_select_topk, loaded from libinfllm.so).
// Rows of the step's shapes: 8 kv heads of 987 units (128K) and of 8,155 units
// (1M), k = 32.  Both results are checked against each other (the same strict
// order: larger score first, ties to the lower index; indices ascending), and
// each is timed with HIP events over back-to-back launches.  Prints one JSON
// line per shape; exit status 1 on any mismatch or HIP error.
#include <dlfcn.h>
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

namespace {

constexpr int kThreads = 1024;
constexpr int kMaxN = 8192;  // keys per row held in LDS (64 KiB of 8-byte keys)

__device__ __forceinline__ uint32_t order_key(float x) {
  if (x != x) return 0u;
  if (x == 0.0f) x = 0.0f;
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// One workgroup per row: keys (order_key(score) << 32 | ~index) padded with 0 to
// the power of two N, sorted descending by the bitonic network (one barrier per
// stage), then the first k indices written ascending (each of the first k threads
// ranks its index among the k by counting).
__global__ void __launch_bounds__(kThreads) bitonic_topk(const float* __restrict__ scores, int n, int n_pow2, int k,
                                                         int32_t* __restrict__ idx) {
  __shared__ uint64_t key[kMaxN];
  __shared__ int32_t top[64];
  const float* s = scores + (int64_t)blockIdx.x * n;
  for (int i = threadIdx.x; i < n_pow2; i += kThreads)
    key[i] = i < n ? ((uint64_t)order_key(s[i]) << 32) | (uint32_t)(~(uint32_t)i) : 0ull;
  __syncthreads();
  for (int size = 2; size <= n_pow2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int p = threadIdx.x; p < n_pow2 / 2; p += kThreads) {
        const int lo = 2 * stride * (p / stride) + (p % stride), hi = lo + stride;
        const bool desc = (lo & size) == 0;  // the sequence's direction in this merge
        const uint64_t a = key[lo], b = key[hi];
        if ((a < b) == desc) {
          key[lo] = b;
          key[hi] = a;
        }
      }
      __syncthreads();
    }
  }
  if (threadIdx.x < k) top[threadIdx.x] = (int32_t)(~(uint32_t)key[threadIdx.x]);
  __syncthreads();
  if (threadIdx.x < k) {
    const int me = top[threadIdx.x];
    int rank = 0;
    for (int j = 0; j < k; ++j) rank += top[j] < me;
    idx[(int64_t)blockIdx.x * k + rank] = me;
  }
}

#define CHECK(x)                                                                  \
  do {                                                                            \
    hipError_t e_ = (x);                                                          \
    if (e_ != hipSuccess) {                                                       \
      std::fprintf(stderr, "HIP error %s at %s:%d\n", hipGetErrorString(e_), __FILE__, __LINE__); \
      std::exit(1);                                                               \
    }                                                                             \
  } while (0)

typedef int (*select_fn)(int32_t, const float*, int32_t, int32_t, int32_t*, void*);

}  // namespace

int main(int argc, char** argv) {
  const char* lib = argc > 1 ? argv[1] : "libinfllm.so";
  void* h = dlopen(lib, RTLD_NOW);
  if (h == nullptr) {
    std::fprintf(stderr, "cannot load %s: %s\n", lib, dlerror());
    return 1;
  }
  select_fn radix = (select_fn)dlsym(h, "infllm_select_topk");
  if (radix == nullptr) return 1;
  const int rows = 8, k = 32, reps = 200;
  for (int n : {987, 8155}) {
    int n_pow2 = 1;
    while (n_pow2 < n) n_pow2 <<= 1;
    std::vector<float> host((size_t)rows * n);
    std::mt19937 gen(n);
    std::normal_distribution<float> nd(0.f, 30.f);
    for (auto& x : host) x = nd(gen);
    float* d_s;
    int32_t *d_a, *d_b;
    CHECK(hipMalloc(&d_s, host.size() * sizeof(float)));
    CHECK(hipMalloc(&d_a, rows * k * sizeof(int32_t)));
    CHECK(hipMalloc(&d_b, rows * k * sizeof(int32_t)));
    CHECK(hipMemcpy(d_s, host.data(), host.size() * sizeof(float), hipMemcpyHostToDevice));
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    float ms_bitonic = 0.f, ms_radix = 0.f;
    for (int pass = 0; pass < 2; ++pass) {  // pass 0 warms up
      CHECK(hipEventRecord(e0, nullptr));
      for (int r = 0; r < reps; ++r)
        hipLaunchKernelGGL(bitonic_topk, dim3(rows), dim3(kThreads), 0, nullptr, d_s, n, n_pow2, k, d_a);
      CHECK(hipGetLastError());
      CHECK(hipEventRecord(e1, nullptr));
      CHECK(hipEventSynchronize(e1));
      CHECK(hipEventElapsedTime(&ms_bitonic, e0, e1));
      CHECK(hipEventRecord(e0, nullptr));
      for (int r = 0; r < reps; ++r)
        if (radix(rows, d_s, n, k, d_b, nullptr) != 0) return 1;
      CHECK(hipEventRecord(e1, nullptr));
      CHECK(hipEventSynchronize(e1));
      CHECK(hipEventElapsedTime(&ms_radix, e0, e1));
    }
    std::vector<int32_t> a(rows * k), b(rows * k);
    CHECK(hipMemcpy(a.data(), d_a, a.size() * 4, hipMemcpyDeviceToHost));
    CHECK(hipMemcpy(b.data(), d_b, b.size() * 4, hipMemcpyDeviceToHost));
    const bool same = std::memcmp(a.data(), b.data(), a.size() * 4) == 0;
    std::printf("{\"n_units\": %d, \"rows\": %d, \"k\": %d, \"bitonic_us\": %.2f, \"radix_us\": %.2f, \"same\": %s}\n", n,
                rows, k, 1e3f * ms_bitonic / reps, 1e3f * ms_radix / reps, same ? "true" : "false");
    CHECK(hipFree(d_s));
    CHECK(hipFree(d_a));
    CHECK(hipFree(d_b));
    if (!same) return 1;
  }
  return 0;
}
