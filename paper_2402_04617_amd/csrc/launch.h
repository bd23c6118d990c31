// Host-side launchers of the gfx950 kernels (internal to the library).  The C ABI
// in abi.cpp validates every argument, then calls these; each returns the
// hipError_t of its launch(es).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.h"

namespace infllm {

// Variable-length batches: sequence b has its own past length past[b] (all
// sequences append the same number of tokens).  Kernels derive each sequence's
// step geometry from it with the host's partition arithmetic.
constexpr int kMaxVarBatch = 64;
struct VarLen {
  int32_t on;
  int64_t past[kMaxVarBatch];
};

// Memory parts of a step split by the positional remap: the memory keys' share
// of `parts`, at least one part per non-empty region.
__host__ __device__ inline int split_parts_mem(int parts, int64_t mem_len, int64_t n_virtual) {
  if (mem_len <= 0 || parts < 2) return 0;
  int pm = (int)((parts * mem_len + n_virtual / 2) / n_virtual);
  return pm < 1 ? 1 : (pm > parts - 1 ? parts - 1 : pm);
}

// Step geometry of a sequence with past length `past` (the partition of
// Section 3.1): `base` supplies the shared fields (l_bs, l_I, k_m, l_X).
__host__ __device__ inline StepGeom seq_geom(const StepGeom& base, int n_local, int64_t past) {
  StepGeom g = base;
  g.n_init = (int32_t)(past < base.unit_base ? past : base.unit_base);
  const int64_t evicted = past - base.unit_base - n_local;
  const int64_t nu = evicted > 0 ? evicted / base.block_size : 0;
  g.n_units = (int32_t)nu;
  g.n_sel = (int32_t)(base.idx_stride < nu ? base.idx_stride : nu);
  g.local_begin = g.n_init + nu * base.block_size;
  g.past_len = past;
  g.n_virtual = (int32_t)(g.n_init + (int64_t)g.n_sel * base.block_size + (past - g.local_begin) + base.n_q);
  return g;
}

// Width of the dimension slices whose partial representative scores the append
// stores (rpart holds D / kRpartDims float64 values per token).
constexpr int kRpartDims = 8;

struct AppendArgs {
  int batch, n_q_heads, n_kv_heads, head_dim, n_q, ring, n_init, n_local;
  int64_t past_len, capacity, q_head_stride, kv_head_stride;
  const void* q;
  const void* k_src;
  const void* v_src;
  void* k_store;
  void* v_store;
  double* qprefix;
  double* rpart;  // [B*Hkv][D/kRpartDims][ring] partial representative scores
  void* k_rot;    // positional remap: keys rotated to their own positions (same layout as k_store)
  RopeArgs rope;
  VarLen var;      // per-sequence past lengths (var.on), else past_len for all
  bool mean_repr;  // units scored by their mean key: no query ring, no representative scores
  bool bf16;
};
// Past length of sequence b of an append.
__host__ __device__ inline int64_t seq_past(const AppendArgs& a, int b) { return a.var.on ? a.var.past[b] : a.past_len; }
struct BuildArgs;
int score_qbar_parts(int G, int n_q);
// qbar: optional float32 output of the chunk's group-query sums: [batch*Hkv][D]
// (the scan total), or with the mean representation [batch*Hkv][parts][D]
// partial sums, parts = score_qbar_parts(G, n_q).
// fused_build: optional unit construction carried by the same launch (its ring
// reads must not overlap the chunk's new ring slots).
hipError_t launch_append(const AppendArgs& a, hipStream_t s, float* qbar, const BuildArgs* fused_build);

struct BuildArgs {
  int batch, n_q_heads, n_kv_heads, head_dim, n_init, n_local, block_size, n_repr;
  int first_unit, n_new, max_units, ring;
  int64_t capacity;
  const void* k_store;
  const double* rpart;
  int32_t* repr_idx;
  float* unit_ksum;
  double* repr_score;  // nullable
  bool mean_repr;      // unit_ksum = mean of the unit's l_bs keys (no representatives)
  // Variable-length batches: sequence b builds units [first[b], first[b] + count[b])
  // (var_on); otherwise every sequence builds [first_unit, first_unit + n_new).
  int32_t var_on;
  int32_t var_first[kMaxVarBatch];
  int32_t var_count[kMaxVarBatch];
  bool bf16;
};
hipError_t launch_build_units(const BuildArgs& a, hipStream_t s);

struct ScoreArgs {
  int batch, n_q_heads, n_kv_heads, head_dim, n_q, n_units, max_units;
  int64_t q_head_stride;
  const void* q;
  const float* unit_ksum;
  float* scores;
  float* qbar_parts;  // workspace
  RopeArgs rope;      // positional remap: the query sum is turned by R(l_L)
  // Variable-length batches: sequence b scores var_units[b] units, rows of
  // `scores` strided by score_stride (var_on); otherwise n_units each, stride n_units.
  int32_t var_on;
  int32_t var_units[kMaxVarBatch];
  int32_t score_stride;
  bool bf16;
};
int score_qbar_parts(int G, int n_q);
hipError_t launch_score(const ScoreArgs& a, hipStream_t s);
// Scoring when a.qbar_parts already holds the query sums as `parts` partials.
hipError_t launch_score_given_qbar(const ScoreArgs& a, int parts, hipStream_t s);

hipError_t launch_select_topk(int rows, const float* scores, int n_units, int k, int32_t* idx,
                              hipStream_t s);
// Rows of different lengths: row r holds row_n[r / rows_per_seq] scores at stride
// `stride`; n_max bounds them.
struct TopkRows {
  int32_t rows_per_seq;
  int32_t row_n[kMaxVarBatch];
};
hipError_t launch_select_topk_var(int rows, const float* scores, int stride, int n_max, const TopkRows& tr, int k,
                                  int32_t* idx, hipStream_t s);

// Query rows per workgroup of the bf16 matrix-core attention kernel, and the
// workgroup count the part chooser aims for (one per compute unit).
constexpr int kMfmaRowsPerWg = 256;
constexpr int kMfmaTargetWgs = 256;
// Workgroups the bf16 decode kernel aims for (two per compute unit), and the
// fewest keys it gives one workgroup.
constexpr int kDecodeTargetWgs = 512;
constexpr int kDecodeMinKeysPerWg = 256;
// Most selected units the decode kernel stages in LDS; longer lookups decode on
// the matrix-core kernel.
constexpr int kDecodeMaxSel = 1024;

// Score rows the matrix-core attention selects from itself: rows of at most
// kFusedSelectShort units hold two keys per thread, longer rows up to
// kFusedSelectMax sixteen (filtered first); at most kFusedSelectMaxK units are
// looked up.
constexpr int kFusedSelectShort = 1024;
constexpr int kFusedSelectMax = 8192;
constexpr int kFusedSelectMaxK = 1024;

struct AttendArgs {
  int batch, n_q_heads, n_kv_heads, head_dim;
  int64_t capacity, q_head_stride, out_head_stride;
  float sm_scale;
  StepGeom geom;
  const void* q;
  const void* k_store;
  const void* v_store;
  // Positional remap: parts [0, parts_mem) cover the memory keys (virtual
  // indices [0, mem_len): I and the selected units) with unrotated keys from
  // k_store and queries turned by R(l_L); parts [parts_mem, parts) cover L and X
  // with keys from k_rot and queries at their own positions.  Without the remap
  // parts_mem = 0 and every part reads k_store.
  const void* k_rot;
  int parts_mem;
  int mem_len;
  RopeArgs rope;
  // Variable-length batches (var.on): each sequence's geometry, memory length and
  // memory parts are derived from var.past[b] (n_local is l_L); geom, mem_len and
  // parts_mem then only carry the shared fields.
  VarLen var;
  int n_local;
  const int32_t* idx;
  // Lookup inside the attention (sel_scores non-null; matrix-core kernel,
  // n_units <= kFusedSelectMax, n_sel <= kFusedSelectMaxK): a workgroup whose tiles hold unit
  // keys selects its kv head's n_sel units from the score row itself, with the
  // select of infllm_select_topk, instead of reading idx; the workgroup of row
  // tile 0 and part 0 also writes the row to idx_out (the -1 padding included).
  const float* sel_scores;  // [batch * n_kv_heads][sel_stride]
  int64_t sel_stride;
  int sel_units;            // most units in any score row (picks the select's keys per thread)
  int32_t* idx_out;         // [batch * n_kv_heads][geom.idx_stride]
  // Per-tile unit-mass partials (with sel_scores; null: off): for tile u of the
  // looked-up units (u < n_sel * l_bs / 64; l_I and l_bs multiples of 64) and
  // attention row r (query-major, r = i * G + h) of kv row bg:
  // mass_part[(bg * mass_tiles + u) * G * n_q + r] = (sum of P over the tile, m)
  // with P = exp2(z * log2(e) - m), z the logit.
  float2* mass_part;
  int mass_tiles;  // tiles per kv row in mass_part (k * l_bs / 64)
  void* out;     // final output (one part)
  float* lse;    // nullable
  // Split-key partials (parts > 1), see the layout in common.h: float32 rows for
  // float32 inputs; for bf16 inputs fp16 rows scaled by 2^-part_exp[row].
  void* part_o;        // [parts][rows][D]
  float* part_lse;     // [parts][rows]
  int32_t* part_exp;   // [parts][rows] (bf16 only)
  int parts;
  bool bf16;
};
// The step of sequence b as a kernel sees it.
struct SeqStep {
  StepGeom geom;
  int mem_len;
  int parts_mem;
};
__host__ __device__ inline SeqStep seq_step(const AttendArgs& a, int b) {
  SeqStep r;
  if (!a.var.on) {
    r.geom = a.geom;
    r.mem_len = a.mem_len;
    r.parts_mem = a.parts_mem;
    return r;
  }
  r.geom = seq_geom(a.geom, a.n_local, a.var.past[b]);
  r.mem_len = r.geom.n_init + r.geom.n_sel * r.geom.block_size;
  r.parts_mem = a.rope.on ? split_parts_mem(a.parts, r.mem_len, r.geom.n_virtual) : 0;
  return r;
}
// Number of key parts the attention uses for this shape, limited by max_parts.
int attend_choose_parts(bool bf16, int batch, int n_q_heads, int n_kv_heads, int n_q, int n_sel, int n_virtual,
                        int max_parts);
hipError_t launch_attend(const AttendArgs& a, hipStream_t s);
// Whether launch_attend runs the matrix-core kernel for these arguments.
bool attend_uses_mfma(const AttendArgs& a);

struct MergeArgs {
  int rows, head_dim, parts, n_q, n_q_heads;
  int64_t out_head_stride;
  const void* part_o;
  const float* part_lse;
  const int32_t* part_exp;
  void* out;
  float* lse;
  bool bf16;
};
hipError_t launch_merge(const MergeArgs& a, hipStream_t s);

// Attention mass of the looked-up units and the frequency-score update.
constexpr int kMassMaxK = 1024;  // most lookup slots per row
struct MassArgs {
  int rows;  // batch * n_kv_heads
  int n_q_heads, n_kv_heads, head_dim;
  int n_q, k, n_units, max_units, block_size;
  int64_t n_init;  // l_I: first position of unit 0
  int64_t capacity, q_head_stride;
  float sm_scale, decay;
  const void* q;
  const void* k_store;
  const int32_t* idx;  // [rows][k]
  const float* lse;    // [batch][Hq][n_q] natural log
  float* mass;         // [rows][k]
  float* freq;         // [rows][max_units] or null
  RopeArgs rope;
  bool bf16;
};
hipError_t launch_unit_mass(const MassArgs& a, hipStream_t s);

// Unit masses from the attention's per-tile partials (AttendArgs::mass_part):
// for slot j < n_sel of kv row bg, mass = sum over the unit's tiles and the
// G * n_q rows of P_sum * exp2(m - lse * log2(e)), lse the step's merged
// natural-log normaliser; slots past n_sel get 0.  The frequency scores as in
// launch_unit_mass.
struct MassPartsArgs {
  int rows;  // batch * n_kv_heads
  int n_q_heads, n_kv_heads, n_q, k, n_sel, n_units, max_units;
  int tiles_per_unit, mass_tiles;
  float decay;
  const float2* mass_part;
  const int32_t* idx;  // [rows][k]
  const float* lse;    // [batch][Hq][n_q]
  float* mass;         // [rows][k]
  float* freq;         // [rows][max_units] or null
};
hipError_t launch_unit_mass_parts(const MassPartsArgs& a, hipStream_t s);

}  // namespace infllm
