/*
 * infllm.h - C ABI of the block-memory attention step of InfLLM
 * (arXiv 2402.04617, "InfLLM: Training-Free Long-Context Extrapolation for LLMs
 * with an Efficient Context Memory"), for AMD Instinct MI355X (gfx950).
 *
 * One attention layer processes a stream in steps (Section 3.1).  A step has
 * past key-values P (length l_P) and current tokens X (length l_X: the chunk size
 * while encoding, 1 while decoding).  P splits into initial tokens I (the first
 * l_I), local tokens L (the last l_L) and evicted tokens E between them.  E is cut
 * into memory units of l_bs tokens; each unit is represented by its r_k tokens of
 * highest representative score r_m (Section 3.2).  Each step scores every unit
 * against X, loads the k_m best, and attends over Concat(I, units, L, X) with one
 * softmax, causal inside X.
 *
 * Conventions for every call
 *  - Every pointer argument except the params/memory structs and the partition
 *    outputs is DEVICE memory owned by the caller.  The library never allocates,
 *    frees or retains memory, and keeps no state between calls.
 *  - Tensors are dense row-major, innermost dimension contiguous, 16-byte aligned.
 *    "dtype" tensors are bfloat16 (INFLLM_BF16) or float32 (INFLLM_F32).
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL = the
 *    default stream).  Device faults surface at the caller's next synchronize.
 *  - Arguments are validated on the host before anything is enqueued; on any
 *    error status nothing is enqueued and no output is touched.  A failed launch
 *    returns INFLLM_E_LAUNCH.  No C++ exception crosses this interface.
 *  - Calls on different streams that write the same buffers race; calls are
 *    otherwise re-entrant.
 *  - All sequences of a batch share one past length, except in
 *    infllm_step_varlen.
 */
#ifndef INFLLM_H
#define INFLLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  INFLLM_OK = 0,
  INFLLM_E_NULL = 1,        /* a required pointer is NULL */
  INFLLM_E_SHAPE = 2,       /* inconsistent sizes or parameters */
  INFLLM_E_RANGE = 3,       /* positions, units or ring slots outside what the memory holds */
  INFLLM_E_UNSUPPORTED = 4, /* valid request this build does not implement (e.g. head_dim) */
  INFLLM_E_WORKSPACE = 5,   /* workspace smaller than required */
  INFLLM_E_LAUNCH = 6,      /* a kernel launch failed */
  INFLLM_E_DEVICE = 7       /* the current device is not a usable gfx950 GPU */
} infllm_status;

typedef enum { INFLLM_F32 = 0, INFLLM_BF16 = 1 } infllm_dtype;

/* Unit representation (Section 3.2): the r_k representative tokens of highest
 * representative score (the method), or the mean of all l_bs keys of the unit
 * (the "Mean Repr" alternative the paper evaluates in its ablation, Section 4). */
typedef enum { INFLLM_REPR_TOKENS = 0, INFLLM_REPR_MEAN = 1 } infllm_repr_mode;

/* Method parameters (Sections 3.1-3.2; the paper's symbols in comments). */
typedef struct {
  int32_t n_q_heads;  /* Hq: query heads; Hq % Hkv == 0.  Query head h reads kv head h / (Hq/Hkv). */
  int32_t n_kv_heads; /* Hkv */
  int32_t head_dim;   /* D: 64 or 128 */
  int32_t n_init;     /* l_I >= 0: initial tokens always attended */
  int32_t n_local;    /* l_L >= 1: local window */
  int32_t block_size; /* l_bs in [1, 256]: tokens per memory unit */
  int32_t n_repr;     /* r_k in [1, l_bs]: representative tokens per unit */
  int32_t topk;       /* k_m >= 0: units loaded per step */
  int32_t dtype;      /* infllm_dtype of q, k, v and the attention output */
  float sm_scale;     /* softmax logit scale > 0 (1 when q or k arrive pre-scaled) */
  /* Positional remap (Section 3.2, "Positional Encoding").  NULL: q and k arrive
   * with their positions already applied and nothing is rotated.  Otherwise a HOST
   * array of D/2 finite rotary angular frequencies theta_i >= 0 (radians per
   * position), read during each call: q and k arrive without positions, dimension
   * pair i = (2i, 2i+1) turns by p*theta_i, and the library applies the remap:
   *  - keys of I and of the memory units are met at distance l_L from every current
   *    token: logit sm_scale * (R(l_L) q) . k, the key unrotated;
   *  - keys of L and X keep their true positions: sm_scale * (R(p_q) q) . (R(t) k_t);
   *  - unit relevance uses the memory distance, sim = (R(l_L) Qbar) . Kbar;
   *  - representative scores are those of the local window, q_{m+j} and k_m at
   *    their own positions.
   * Half-split pairs (i, i + D/2) are the same model after one fixed permutation
   * of the head dimensions of q and k.  Needs memory.k_rot. */
  const double* rope_inv_freq;
  /* infllm_repr_mode.  With INFLLM_REPR_MEAN a unit is scored by the mean of its
   * keys, sim(X, B) = sum_i q_{i+l_P} . mean_j k_j^B: unit_ksum holds that mean,
   * repr_idx is neither written nor needed, n_repr is ignored, and no
   * representative scores are formed, so qprefix and rpart are not used (NULL
   * allowed) and the append only stores K and V. */
  int32_t repr_mode;
} infllm_params;

/*
 * The layer's context memory, all device memory owned by the caller.
 *   k, v       [batch][Hkv][capacity][D] dtype.  Token-ordered store of P (and of X
 *              once appended): I, the units and L are views of it, so eviction
 *              moves no data.
 *   repr_idx   [batch][Hkv][max_units][r_k] int32: offsets inside the unit of its
 *              representative tokens R(B), ascending.  Written by infllm_build_units.
 *   unit_ksum  [batch][Hkv][D/4][max_units][4] float32: per unit, the sum of its
 *              representative keys, sum_{j in R(B)} k_j, stored four dimensions per
 *              16-byte cell, unit-contiguous (the layout unit scoring streams; with
 *              max_units a multiple of 8 and a 128-byte aligned base every row
 *              starts on a cache line, which scoring reads 64 units at a time).
 *   qprefix    [batch][Hkv][ring][D] float64 ring: slot (t mod ring) holds
 *              sum_{p <= t} sum_{h in group} q^h_p, the running sum of the group's
 *              queries.  Written and read by infllm_append.
 *   rpart      [batch][Hkv][D/8][ring] float64 ring: slot (t mod ring) of row s
 *              holds sum over dims d in [8s, 8s+8) of k_t[d] * W_t[d], where
 *              W_t = qprefix(t + l_L) - qprefix(t) is the window query sum of token
 *              t; summed over s it is l_L*G times the representative score r_t of
 *              Section 3.2.  Written by infllm_append once position t + l_L is
 *              appended, read by infllm_build_units.
 *   k_rot      [batch][Hkv][capacity][D] dtype, only with the positional remap
 *              (params.rope_inv_freq set; may be NULL otherwise): every key rotated
 *              to its own position, R(t) k_t, written by infllm_append next to the
 *              unrotated k; the attention reads L and X from it.
 * Unit b of E covers positions [l_I + b*l_bs, l_I + (b+1)*l_bs).
 * For bf16 the attention entry points need one [capacity][D] slice of k or v to
 * span at most 4 GiB (capacity * D * 2 bytes; 16M tokens at D = 128), else
 * INFLLM_E_UNSUPPORTED.
 */
typedef struct {
  int32_t batch;
  int64_t capacity;
  void* k;
  void* v;
  int32_t max_units;
  int32_t* repr_idx;
  float* unit_ksum;
  double* qprefix;
  double* rpart;
  int32_t ring;
  void* k_rot;
} infllm_memory;

/* Partition of P at past length l_P (Section 3.1): |I| = min(l_I, l_P);
 * n_units = floor((l_P - l_I - l_L) / l_bs) whole units (0 if negative);
 * L = [local_begin, l_P) with local_begin = |I| + n_units*l_bs.  Evicted tokens
 * that do not fill a whole unit stay in L.  Host only; outputs are host pointers. */
infllm_status infllm_partition(const infllm_params* p, int64_t past_len, int64_t* n_init,
                               int32_t* n_units, int64_t* local_begin);

/* Bytes of device workspace that infllm_score_units, infllm_chunk_attend and the
 * step calls need for `batch` sequences and n_q current tokens (split-key
 * partial results and query sums, plus the per-tile unit-mass partials that
 * infllm_step_mass keeps at the end of its workspace).  Depends only on these
 * arguments. */
size_t infllm_workspace_bytes(const infllm_params* p, int32_t batch, int32_t n_q);
/* The same size under the name the attention's callers may know it by; both names
 * cover every call that takes a workspace (scoring as well as attention). */
size_t infllm_attend_workspace_bytes(const infllm_params* p, int32_t batch, int32_t n_q);

/* Append the current tokens X at positions [past_len, past_len + n_q).
 *  q: [batch][Hq] heads of n_q x D dtype rows; head h of sequence b starts at
 *     q + (b*Hq + h)*q_head_stride elements (q_head_stride >= n_q*D).
 *  k, v: chunk keys/values laid out the same way with kv_head_stride; both NULL
 *     when the caller has already written them into the store.
 * Copies k, v into the store (and, with the positional remap, the rotated keys
 * into k_rot; the ring then sums the group's queries rotated to their positions),
 * extends the qprefix ring and, for every appended
 * position p with t = p - l_L >= l_I, writes the partial representative scores of
 * token t into rpart (what the representative score r_t of Section 3.2 needs
 * once t is evicted).  Positions must be appended in order: slot (past_len - 1)
 * must hold the running sum through past_len - 1.  E_RANGE if past_len + n_q >
 * capacity, or if the ring would lose the running sum of a token t before its
 * scores are formed (it needs ring >= l_L + n_q in steady streaming); E_NULL if
 * such a token lies inside the chunk (l_L < n_q) and k is NULL. */
infllm_status infllm_append(const infllm_params* p, const infllm_memory* m, const void* q,
                            int64_t q_head_stride, const void* k, const void* v,
                            int64_t kv_head_stride, int32_t n_q, int64_t past_len, void* stream);

/* Memory-unit construction (Section 3.2, "Block-Level Memory Units").
 * For units [first_unit, first_unit + n_new) of every (sequence, kv head):
 * r_m = 1/(l_L*G) * sum_{h in group} sum_{j=1..l_L} q^h_{m+j} . k_m for each of its
 * l_bs tokens (G = Hq/Hkv), then R(B) = the r_k tokens of largest r_m (ties: lower
 * position).  r_m is the sum of the rpart rows that infllm_append wrote for m.
 * Writes repr_idx and unit_ksum.  `past_len` is the number of positions appended
 * so far; every window m+1..m+l_L must lie below it and the ring must still hold
 * the unit's slots, first_pos >= past_len - ring (E_RANGE otherwise).
 * repr_score: optional [batch][Hkv][n_new][l_bs] float64 output of r_m. */
infllm_status infllm_build_units(const infllm_params* p, const infllm_memory* m, int32_t first_unit,
                                 int32_t n_new, int64_t past_len, double* repr_score, void* stream);

/* Unit relevance (Section 3.2, "memory lookup"):
 * sim(X, B) = sum_{i=1..l_X} sum_{j=1..r_k} q_{i+l_P} . k_{b_j}, one score per
 * (sequence, kv head, unit) with the query side summed over the kv head's query
 * group.  q as in infllm_append.  scores: [batch][Hkv][n_units] float32.
 * n_units must not exceed max_units.  Needs the workspace. */
infllm_status infllm_score_units(const infllm_params* p, const infllm_memory* m, const void* q,
                                 int64_t q_head_stride, int32_t n_q, int32_t n_units, float* scores,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* Top-k lookup f(X, E) (Section 3.2): for each of `rows` rows of `scores`
 * ([rows][n_units] float32), the min(k, n_units) largest, ties to the lower index,
 * written ascending to idx [rows][k] int32 followed by -1 padding.  NaN scores
 * rank below every number; -0 equals +0.  The selection depends on nothing but
 * the scores and k, so it takes no params struct (rows = batch * Hkv for the
 * scores infllm_score_units writes; k is k_m). */
infllm_status infllm_select_topk(int32_t rows, const float* scores, int32_t n_units, int32_t k,
                                 int32_t* idx, void* stream);

/* Attention of the current tokens over the current key-value cache (Section 3.1):
 * O = Attn[Q X, Concat(C_k, K X), Concat(C_v, V X)] with C = Concat(I, f(X,E), L).
 * For query i of head h (kv head g = h / G), one softmax of sm_scale * q . k over
 * I, the units idx[b][g][0 .. min(k, n_units)) (entries that are negative or
 * >= n_units are skipped), L, and X positions past_len .. past_len + i.
 * The chunk's K/V must already be in the store.
 *  out: [batch][Hq] heads of n_q x D dtype rows, head stride out_head_stride.
 *  lse: optional [batch][Hq][n_q] float32 natural-log sum of exp of the logits.
 * The keys are split into parts processed in parallel whose partial softmaxes are
 * merged by their log-sum-exp; the workspace holds the partials.  With the
 * positional remap, memory keys and local keys always fall in different parts,
 * so the workspace is required whenever I or a unit is attended (E_WORKSPACE). */
infllm_status infllm_chunk_attend(const infllm_params* p, const infllm_memory* m, const void* q,
                                  int64_t q_head_stride, int32_t n_q, int64_t past_len,
                                  const int32_t* idx, int32_t k, void* out, int64_t out_head_stride,
                                  float* lse, void* workspace, size_t workspace_bytes, void* stream);

/* The two halves of infllm_chunk_attend, for callers that time or schedule them
 * apart.  infllm_attend_partial writes per-part normalised outputs and lse into the
 * workspace and reports the part count; infllm_lse_merge combines them
 * (LSE = log sum_s exp(lse_s), O = sum_s exp(lse_s - LSE) O_s) into out / lse.
 * With one part, infllm_attend_partial writes out and lse directly and
 * infllm_lse_merge must not be called.  Arguments as in infllm_chunk_attend.
 * Workspace layout of the partials (rows = batch*Hq*n_q): [n_parts][rows][D]
 * values, then [n_parts][rows] float32 lse, then for bf16 inputs [n_parts][rows]
 * int32 exponents e.  Float32 inputs store float32 values; bf16 inputs store each
 * part's row as fp16 values v with O_s = v * 2^e, e chosen per row so that its
 * largest magnitude lies in [2^14, 2^15) (11-bit precision relative to it). */
infllm_status infllm_attend_partial(const infllm_params* p, const infllm_memory* m, const void* q,
                                    int64_t q_head_stride, int32_t n_q, int64_t past_len,
                                    const int32_t* idx, int32_t k, void* out, int64_t out_head_stride,
                                    float* lse, void* workspace, size_t workspace_bytes,
                                    int32_t* n_parts, void* stream);
infllm_status infllm_lse_merge(const infllm_params* p, int32_t batch, int32_t n_q, int32_t n_parts,
                               const void* workspace, size_t workspace_bytes, void* out,
                               int64_t out_head_stride, float* lse, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): infllm_chunk_attend with
 * no workspace argument.  The split-key partials go to a device array the library
 * owns, INFLLM_NOALLOC_SCRATCH_BYTES (32 MiB) on every GPU it runs on, held from
 * the library's load until the process ends; nothing is allocated or freed by the
 * call.  The part count is chosen to fit that array: E_WORKSPACE when even the
 * fewest parts the call needs do not fit (batch*Hq*n_q rows of D*2 + 8 bytes per
 * part for bf16, (D + 1)*4 for float32; two parts whenever the positional remap
 * attends I or a unit).  All calls on one GPU share the array and every call
 * rewrites what it reads of it (nothing in it needs clearing), so such calls that
 * overlap on one GPU (different streams, no ordering between them) race.
 * E_DEVICE if the array's address cannot be looked up on the current device.
 * Otherwise as infllm_chunk_attend, whose results it reproduces when both use the
 * same number of key parts. */
#define INFLLM_NOALLOC_SCRATCH_BYTES (32u << 20)
infllm_status infllm_chunk_attend_noalloc(const infllm_params* p, const infllm_memory* m, const void* q,
                                          int64_t q_head_stride, int32_t n_q, int64_t past_len,
                                          const int32_t* idx, int32_t k, void* out, int64_t out_head_stride,
                                          float* lse, void* stream);

/* Attention mass of the looked-up units and the frequency score of the cache
 * policy (Section 3.2, "Cache Management", and the appendix on the cache
 * management strategy: s_b = s_b * d + sum_{j<l_X} sum_{i in b} attention score).
 * For the step at past_len with current tokens X (n_q of them, queries q as given
 * to the attention) and its lookup idx [batch][Hkv][k] (as infllm_select_topk
 * writes it: distinct entries, -1 padding):
 *   mass [batch][Hkv][k] float32 (required when k > 0): for slot j with unit
 *        b = idx[..][j] in [0, n_units(past_len)), the softmax probability the step's
 *        attention gave b's l_bs keys, summed over the n_q queries and the G query
 *        heads of the kv group: sum_h sum_i sum_{t in b} exp(z - lse) with z the
 *        attention logit (under the positional remap the query turned by R(l_L)),
 *        so it lies in [0, G*n_q]; 0 for a -1 or out-of-range entry;
 *   lse  [batch][Hq][n_q] float32: the step's natural-log normaliser, as
 *        infllm_chunk_attend / infllm_step write it (required when n_q, k > 0);
 *   freq [batch][Hkv][max_units] float32, nullable, read and written: the
 *        frequency score of every built unit b < n_units(past_len) becomes
 *        freq * decay + mass(b), with mass 0 for units not looked up (all units
 *        stay resident here, so all of them decay).  Zero it before the first step.
 * decay: finite, >= 0 (the paper uses 0.1).  Run it after the step's attention on
 * the same stream.  All sequences share past_len (for a batch stepped with
 * infllm_step_varlen, call it per sequence on a one-sequence view of the memory).
 * E_UNSUPPORTED for k > 1024. */
infllm_status infllm_unit_mass(const infllm_params* p, const infllm_memory* m, const void* q,
                               int64_t q_head_stride, int32_t n_q, int64_t past_len, const int32_t* idx, int32_t k,
                               const float* lse, float decay, float* mass, float* freq, void* stream);

/* One whole step of the layer (Sections 3.1-3.2) for the current tokens X at
 * positions [past_len, past_len + n_q), in this order on `stream`:
 *   1. unit construction for units [units_built, n_units(past_len)), the units
 *      evicted since the caller's previous step (as infllm_build_units);
 *   2. append of X (as infllm_append; k, v may be NULL when already stored);
 *   3. relevance of every unit: scores [batch][Hkv][n_units(past_len)] float32;
 *   4. lookup of the k_m best: idx [batch][Hkv][k_m] int32 (as infllm_select_topk);
 *   5. attention (as infllm_chunk_attend) into out / lse.
 * With bf16 chunks (the matrix-core attention), at most 8,192 units and k_m at
 * most 1,024, stages 4 and 5 share one launch: the attention selects the units
 * from the scores itself and writes idx as stage 4 would (same entries, order
 * and padding).
 * units_built is the number of units built by earlier steps (0 for the first
 * step); afterwards n_units(past_len) units are built.  Every stage is validated
 * before the first is enqueued. */
infllm_status infllm_step(const infllm_params* p, const infllm_memory* m, const void* q, int64_t q_head_stride,
                          const void* k, const void* v, int64_t kv_head_stride, int32_t n_q, int64_t past_len,
                          int32_t units_built, float* scores, int32_t* idx, void* out, int64_t out_head_stride,
                          float* lse, void* workspace, size_t workspace_bytes, void* stream);

/* infllm_step followed by the attention mass of its lookup and the frequency
 * score update (Section 3.2, "Cache Management"; the appendix on the cache
 * management strategy): mass [batch][Hkv][k_m] and freq [batch][Hkv][max_units]
 * (nullable) as infllm_unit_mass writes them for this step's q, idx and lse, with
 * the same decay and the same argument rules (lse is required when n_q, k_m > 0).
 * Where the matrix-core attention also selects the units (bf16 chunks, at most
 * 8,192 units, k_m at most 1,024) and l_I and l_bs are multiples of 64, the
 * attention writes each looked-up 64-key tile's per-row sum of P and its running
 * maximum into the end of the workspace, and one small launch after the merge
 * forms the masses from
 * them and the merged lse (no second pass over the keys); otherwise the step is
 * followed by the unit-mass kernel.  The two agree to float32 rounding.
 * infllm_workspace_bytes covers the partials. */
infllm_status infllm_step_mass(const infllm_params* p, const infllm_memory* m, const void* q,
                               int64_t q_head_stride, const void* k, const void* v, int64_t kv_head_stride,
                               int32_t n_q, int64_t past_len, int32_t units_built, float* scores, int32_t* idx,
                               void* out, int64_t out_head_stride, float* lse, float decay, float* mass, float* freq,
                               void* workspace, size_t workspace_bytes, void* stream);

/* One step of a batch whose sequences have different past lengths (a serving
 * batch: each sequence decodes, or encodes a chunk, at its own position).
 * Sequence b appends its n_q tokens at [past_lens[b], past_lens[b] + n_q) and
 * runs the five stages of infllm_step against its own partition; past_lens and
 * units_built are HOST arrays of `batch` entries (units_built[b] as in
 * infllm_step, per sequence).  scores: [batch][Hkv][max_units] float32 (row
 * stride memory.max_units; sequence b fills its first n_units(past_lens[b])
 * entries of each row).  Everything else as in infllm_step.  batch <= 64
 * (E_UNSUPPORTED beyond); each sequence is validated as its own step first. */
infllm_status infllm_step_varlen(const infllm_params* p, const infllm_memory* m, const void* q,
                                 int64_t q_head_stride, const void* k, const void* v, int64_t kv_head_stride,
                                 int32_t n_q, const int64_t* past_lens, const int32_t* units_built, float* scores,
                                 int32_t* idx, void* out, int64_t out_head_stride, float* lse, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* Static description of a status code. */
const char* infllm_status_string(infllm_status s);

#ifdef __cplusplus
}
#endif

#endif /* INFLLM_H */
