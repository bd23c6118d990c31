// Internal helpers shared by the gfx950 kernels of the InfLLM step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace infllm {

typedef uint16_t bf16_t;  // bfloat16 bit pattern as stored in HBM

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kNumXcd = 8;  // MI355X: 8 XCDs, workgroups dispatched round-robin over them

__device__ __forceinline__ float bf16_to_f32(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// Round to nearest even (hardware v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16_t f32_to_bf16(float x) {
  __bf16 h = (__bf16)x;
  return __builtin_bit_cast(bf16_t, h);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ static float load(const float* p) { return *p; }
  __device__ static void store(float* p, float x) { *p = x; }
};
template <> struct Elem<bf16_t> {
  __device__ static float load(const bf16_t* p) { return bf16_to_f32(*p); }
  __device__ static void store(bf16_t* p, float x) { *p = f32_to_bf16(x); }
};

// Geometry of one step's key set, shared by the attention kernels.  The keys a
// query sees are laid out on a "virtual" axis v in [0, n_virtual):
//   [0, n_init)                        initial tokens I          -> position v
//   [n_init, n_init + n_sel*l_bs)      selected units, in idx order
//   [.., n_virtual - n_q)              local tokens L            -> local_begin + ...
//   [n_virtual - n_q, n_virtual)       current tokens X (causal) -> past_len + ...
// L and X are adjacent in the store, so the tail of the axis is one contiguous run.
struct StepGeom {
  int32_t n_init;        // |I|
  int32_t n_units;       // units formed (valid idx values are < n_units)
  int32_t n_sel;         // idx entries used = min(k, n_units)
  int32_t block_size;    // l_bs
  int32_t unit_base;     // l_I: first position of unit 0
  int32_t idx_stride;    // k: idx row stride
  int64_t local_begin;   // first position of L
  int64_t past_len;      // l_P
  int32_t n_q;           // l_X
  int32_t n_virtual;     // total keys on the virtual axis
};

// Store position of virtual key v; -1 for a skipped (invalid) unit entry.
__device__ __forceinline__ int64_t virtual_pos(const StepGeom& g, const int32_t* idx_row, int v) {
  if (v < g.n_init) return v;
  int w = v - g.n_init;
  int sel_len = g.n_sel * g.block_size;
  if (w < sel_len) {
    int u = w / g.block_size;
    int off = w - u * g.block_size;
    int b = idx_row[u];
    if (b < 0 || b >= g.n_units) return -1;
    return (int64_t)g.unit_base + (int64_t)b * g.block_size + off;
  }
  return g.local_begin + (w - sel_len);
}

// Positional remap (Section 3.2, "Positional Encoding"): rotary tables for a
// step whose q and k arrive without positions.  Dimension pair i = (2i, 2i+1)
// turns by the angle p * theta_i.  Keys of I and of the memory units are kept
// unrotated and met by queries turned by R(l_L) (distance l_L); keys of L and X
// are rotated to their own positions and met by queries at theirs.
constexpr int kMaxPairs = 64;  // D/2 at D = 128
struct RopeArgs {
  int32_t on;                // 0: positions pre-applied, nothing is rotated
  double rev[kMaxPairs];     // theta_i / (2 pi): revolutions per position of pair i
  float mem_cos[kMaxPairs];  // cos(l_L theta_i)
  float mem_sin[kMaxPairs];  // sin(l_L theta_i)
};

// cos and sin of p * theta_i.  The angle is reduced to [0, 1) revolutions in
// float64 (p * theta_i reaches 10^6 radians at a million positions); the
// hardware sine and cosine take revolutions.
__device__ __forceinline__ void rope_cos_sin(const RopeArgs& r, int64_t pos, int i, float& c, float& s) {
  double t = (double)pos * r.rev[i];
  t -= floor(t);
  const float f = (float)t;
  s = __builtin_amdgcn_sinf(f);
  c = __builtin_amdgcn_cosf(f);
}

// XCD-aware workgroup order: consecutive logical ids land on the same XCD (and so
// share its L2), given round-robin dispatch of linear ids over the XCDs.
__device__ __forceinline__ int xcd_logical_block(int linear, int total) {
  if (total % kNumXcd != 0) return linear;
  int per = total / kNumXcd;
  return (linear % kNumXcd) * per + linear / kNumXcd;
}

// Split-key partial rows.  A part's normalised output row O_s (a convex
// combination of value rows) is stored, for bfloat16 inputs, as fp16 values
// O_s * 2^-e with one exponent e per row chosen so that the row's largest
// magnitude lands in [2^14, 2^15): every element keeps fp16's 11-bit precision
// relative to that maximum, at half the bytes of float32.  Float32 inputs keep
// float32 rows.
__device__ __forceinline__ int partial_row_exponent(float row_absmax) {
  if (!(row_absmax > 0.f) || row_absmax == __builtin_inff()) return 0;  // zero, NaN or inf: unscaled
  const int eb = (int)((__float_as_uint(row_absmax) >> 23) & 255u);
  const int e = eb - 127 - 14;
  return e < -100 ? -100 : (e > 100 ? 100 : e);
}
__device__ __forceinline__ float exp2_int(int e) { return __uint_as_float((uint32_t)(127 + e) << 23); }  // |e| <= 100
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  const _Float16 a = (_Float16)lo, b = (_Float16)hi;  // round to nearest even
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}
__device__ __forceinline__ float f16_lo(uint32_t w) { return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu)); }
__device__ __forceinline__ float f16_hi(uint32_t w) { return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16)); }

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}
__device__ __forceinline__ double wave_sum_f64(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

}  // namespace infllm
