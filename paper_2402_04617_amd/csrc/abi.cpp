// C ABI of the InfLLM step (declared in include/infllm.h): argument validation on
// the host, partition arithmetic, workspace sizing and kernel dispatch on the
// caller's stream.  Every check runs before the first HIP call, so invalid
// arguments are rejected without touching the device.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <algorithm>
#include <cstring>

#include "../../include/infllm.h"
#include "launch.h"

using namespace infllm;

namespace infllm {
int attend_max_parts(bool bf16, int G, int n_q, int64_t max_virtual);
}

namespace {

constexpr int kMaxDevices = 64;
std::atomic<int> g_device_ok[kMaxDevices];  // 0 unknown, 1 gfx950, 2 unusable

infllm_status check_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return INFLLM_E_DEVICE;
  }
  int st = g_device_ok[dev].load(std::memory_order_relaxed);
  if (st == 0) {
    hipDeviceProp_t prop;
    st = 2;
    if (hipGetDeviceProperties(&prop, dev) == hipSuccess && std::strncmp(prop.gcnArchName, "gfx950", 6) == 0)
      st = 1;
    (void)hipGetLastError();
    g_device_ok[dev].store(st, std::memory_order_relaxed);
  }
  return st == 1 ? INFLLM_OK : INFLLM_E_DEVICE;
}

// Device scratch of infllm_chunk_attend_noalloc: a file-scope array that every GPU
// the library runs on holds from module load until the process ends, in place of a
// caller workspace.  Host code never passes the array's name (a host-side stand-in)
// to a kernel: on first use on a device, with that device current, its device
// address is looked up once and kept per device.
constexpr size_t kScratchBytes = (size_t)INFLLM_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];
std::atomic<void*> g_scratch_ptr[kMaxDevices];

// Device address of `scratch` on the current device (nullptr on failure).
void* scratch_device_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return nullptr;
  }
  void* ptr = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (ptr == nullptr) {
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[dev].store(ptr, std::memory_order_release);
  }
  return ptr;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
int esize(const infllm_params* p) { return p->dtype == INFLLM_BF16 ? 2 : 4; }

infllm_status check_params(const infllm_params* p) {
  if (p == nullptr) return INFLLM_E_NULL;
  if (p->n_q_heads <= 0 || p->n_kv_heads <= 0 || p->n_q_heads % p->n_kv_heads != 0) return INFLLM_E_SHAPE;
  if (p->dtype != INFLLM_F32 && p->dtype != INFLLM_BF16) return INFLLM_E_SHAPE;
  if (p->head_dim <= 0) return INFLLM_E_SHAPE;
  if (p->head_dim != 64 && p->head_dim != 128) return INFLLM_E_UNSUPPORTED;
  if (p->n_init < 0 || p->n_local < 1 || p->block_size < 1 || p->topk < 0) return INFLLM_E_SHAPE;
  if (p->block_size > 256) return INFLLM_E_UNSUPPORTED;
  if (p->n_repr < 1 || p->n_repr > p->block_size) return INFLLM_E_SHAPE;
  if (!std::isfinite(p->sm_scale) || !(p->sm_scale > 0.f)) return INFLLM_E_SHAPE;
  if (p->repr_mode != INFLLM_REPR_TOKENS && p->repr_mode != INFLLM_REPR_MEAN) return INFLLM_E_SHAPE;
  if (p->rope_inv_freq != nullptr) {
    for (int i = 0; i < p->head_dim / 2; ++i)
      if (!std::isfinite(p->rope_inv_freq[i]) || p->rope_inv_freq[i] < 0.0) return INFLLM_E_SHAPE;
  }
  return INFLLM_OK;
}

bool remap(const infllm_params* p) { return p->rope_inv_freq != nullptr; }
// Units scored by their mean key: no representative scores, so no query ring.
bool mean_repr(const infllm_params* p) { return p->repr_mode == INFLLM_REPR_MEAN; }

// Rotary tables of the positional remap, formed in float64 on the host.
RopeArgs rope_args(const infllm_params* p) {
  RopeArgs r;
  std::memset(&r, 0, sizeof(r));
  if (!remap(p)) return r;
  r.on = 1;
  const double two_pi = 6.283185307179586476925286766559;
  for (int i = 0; i < p->head_dim / 2; ++i) {
    const double th = p->rope_inv_freq[i];
    r.rev[i] = th / two_pi;
    r.mem_cos[i] = (float)std::cos((double)p->n_local * th);
    r.mem_sin[i] = (float)std::sin((double)p->n_local * th);
  }
  return r;
}

infllm_status check_store(const infllm_params* p, const infllm_memory* m) {
  if (m == nullptr || m->k == nullptr || m->v == nullptr) return INFLLM_E_NULL;
  if (m->batch < 1 || m->capacity < 1) return INFLLM_E_SHAPE;
  if (!aligned16(m->k) || !aligned16(m->v)) return INFLLM_E_SHAPE;
  if (remap(p)) {
    if (m->k_rot == nullptr) return INFLLM_E_NULL;
    if (!aligned16(m->k_rot)) return INFLLM_E_SHAPE;
  }
  return INFLLM_OK;
}

infllm_status check_units(const infllm_params* p, const infllm_memory* m) {
  if ((m->repr_idx == nullptr && !mean_repr(p)) || m->unit_ksum == nullptr) return INFLLM_E_NULL;
  if (m->max_units < 0) return INFLLM_E_SHAPE;
  if (!aligned16(m->unit_ksum)) return INFLLM_E_SHAPE;
  return INFLLM_OK;
}

// Rows of `n_q` tokens per head with stride `head_stride` elements, read as 16-byte vectors.
infllm_status check_rows(const infllm_params* p, const void* ptr, int64_t head_stride, int32_t n_q) {
  if (ptr == nullptr) return INFLLM_E_NULL;
  if (head_stride < (int64_t)n_q * p->head_dim) return INFLLM_E_SHAPE;
  if (((head_stride * esize(p)) & 15) != 0 || !aligned16(ptr)) return INFLLM_E_SHAPE;
  return INFLLM_OK;
}

struct Part {
  int64_t n_init, local_begin;
  int32_t n_units;
};
Part partition(const infllm_params* p, int64_t past_len) {
  Part r;
  r.n_init = past_len < p->n_init ? past_len : p->n_init;
  const int64_t evicted = past_len - p->n_init - p->n_local;
  const int64_t nu = evicted > 0 ? evicted / p->block_size : 0;
  r.n_units = (int32_t)(nu > INT32_MAX ? INT32_MAX : nu);
  r.local_begin = r.n_init + nu * p->block_size;
  return r;
}

int64_t max_virtual_keys(const infllm_params* p, int32_t n_q) {
  return (int64_t)p->n_init + (int64_t)p->topk * p->block_size + p->n_local + p->block_size - 1 + n_q;
}

// Workspace bytes of one part's partial row: fp16 values, lse and exponent for
// bf16 inputs; float32 values and lse for float32 inputs.
size_t part_row_bytes(const infllm_params* p) {
  return p->dtype == INFLLM_BF16 ? (size_t)p->head_dim * 2u + 8u : (size_t)(p->head_dim + 1) * 4u;
}

size_t attend_ws_bytes(const infllm_params* p, int32_t batch, int32_t n_q, int parts) {
  const int64_t rows = (int64_t)batch * p->n_q_heads * n_q;
  return (size_t)parts * (size_t)rows * part_row_bytes(p);
}

// Partial arrays inside the workspace: [parts][rows][D] values, then [parts][rows]
// lse, then (bf16) [parts][rows] exponents.
void partial_layout(const infllm_params* p, void* workspace, int parts, int64_t rows, void** o, float** lse,
                    int32_t** ex) {
  const size_t vbytes = (size_t)parts * (size_t)rows * (size_t)p->head_dim * (p->dtype == INFLLM_BF16 ? 2u : 4u);
  char* w = (char*)workspace;
  *o = w;
  *lse = w ? (float*)(w + vbytes) : nullptr;
  *ex = (w && p->dtype == INFLLM_BF16) ? (int32_t*)(w + vbytes + (size_t)parts * (size_t)rows * 4u) : nullptr;
}

size_t qbar_ws_bytes(const infllm_params* p, int32_t batch, int32_t n_q) {
  const int G = p->n_q_heads / p->n_kv_heads;
  return (size_t)batch * p->n_kv_heads * score_qbar_parts(G, n_q) * p->head_dim * 4u;
}

infllm_status launch_status(hipError_t e) {
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return INFLLM_E_LAUNCH;
  }
  return INFLLM_OK;
}

// Shared preparation of infllm_chunk_attend / infllm_attend_partial.
infllm_status prepare_attend(const infllm_params* p, const infllm_memory* m, const void* q,
                             int64_t q_head_stride, int32_t n_q, int64_t past_len, const int32_t* idx,
                             int32_t k, void* out, int64_t out_head_stride, float* lse, void* workspace,
                             size_t workspace_bytes, AttendArgs* a) {
  infllm_status st;
  if ((st = check_params(p)) != INFLLM_OK) return st;
  if ((st = check_store(p, m)) != INFLLM_OK) return st;
  if (n_q < 0 || past_len < 0 || k < 0) return INFLLM_E_SHAPE;
  if (past_len + n_q > m->capacity) return INFLLM_E_RANGE;
  if ((st = check_rows(p, q, q_head_stride, n_q)) != INFLLM_OK) return st;
  if ((st = check_rows(p, out, out_head_stride, n_q)) != INFLLM_OK) return st;
  const Part part = partition(p, past_len);
  const int32_t n_sel = k < part.n_units ? k : part.n_units;
  if (n_sel > 0 && idx == nullptr) return INFLLM_E_NULL;
  const int64_t n_virtual = part.n_init + (int64_t)n_sel * p->block_size + (past_len - part.local_begin) + n_q;
  if (n_virtual > INT32_MAX) return INFLLM_E_UNSUPPORTED;
  const bool bf16 = p->dtype == INFLLM_BF16;
  // the bf16 kernels address one (sequence, kv head) slice of the store with 32-bit byte offsets
  if (bf16 && (uint64_t)m->capacity * (uint64_t)p->head_dim * 2u > 0xFFFFFFFFull) return INFLLM_E_UNSUPPORTED;
  const int64_t rows = (int64_t)m->batch * p->n_q_heads * n_q;
  const size_t per_part = rows > 0 ? (size_t)rows * part_row_bytes(p) : 1;
  const int max_parts = (workspace == nullptr) ? 0 : (int)(workspace_bytes / per_part > 4096 ? 4096 : workspace_bytes / per_part);
  int parts = attend_choose_parts(bf16, m->batch, p->n_q_heads, p->n_kv_heads, n_q, n_sel, (int)n_virtual,
                                  max_parts);
  if (parts < 1) return INFLLM_E_WORKSPACE;
  // With the remap, memory keys (I and the units) and local keys go to
  // different parts, in proportion to their counts.
  const int64_t mem_len = part.n_init + (int64_t)n_sel * p->block_size;
  int parts_mem = 0;
  if (remap(p) && mem_len > 0) {
    if (parts < 2) {
      if (max_parts < 2) return INFLLM_E_WORKSPACE;
      parts = 2;
    }
    parts_mem = split_parts_mem(parts, mem_len, n_virtual);
  }
  if (parts > 1 && !aligned16(workspace)) return INFLLM_E_SHAPE;

  std::memset(a, 0, sizeof(*a));
  a->batch = m->batch;
  a->n_q_heads = p->n_q_heads;
  a->n_kv_heads = p->n_kv_heads;
  a->head_dim = p->head_dim;
  a->capacity = m->capacity;
  a->q_head_stride = q_head_stride;
  a->out_head_stride = out_head_stride;
  a->sm_scale = p->sm_scale;
  a->geom.n_init = (int32_t)part.n_init;
  a->geom.n_units = part.n_units;
  a->geom.n_sel = n_sel;
  a->geom.block_size = p->block_size;
  a->geom.unit_base = p->n_init;
  a->geom.idx_stride = k;
  a->geom.local_begin = part.local_begin;
  a->geom.past_len = past_len;
  a->geom.n_q = n_q;
  a->geom.n_virtual = (int32_t)n_virtual;
  a->q = q;
  a->k_store = m->k;
  a->v_store = m->v;
  a->k_rot = m->k_rot;
  a->parts_mem = parts_mem;
  a->mem_len = (int)mem_len;
  a->rope = rope_args(p);
  a->n_local = p->n_local;
  a->idx = idx;
  a->out = out;
  a->lse = lse;
  a->parts = parts;
  partial_layout(p, workspace, parts, rows, &a->part_o, &a->part_lse, &a->part_exp);
  a->bf16 = bf16;
  return INFLLM_OK;
}

MergeArgs merge_args(const infllm_params* p, int32_t batch, int32_t n_q, int32_t n_parts, const void* workspace,
                     void* out, int64_t out_head_stride, float* lse) {
  MergeArgs ma;
  const int64_t rows = (int64_t)batch * p->n_q_heads * n_q;
  ma.rows = (int)rows;
  ma.head_dim = p->head_dim;
  ma.parts = n_parts;
  ma.n_q = n_q;
  ma.n_q_heads = p->n_q_heads;
  ma.out_head_stride = out_head_stride;
  void* po;
  float* pl;
  int32_t* pe;
  partial_layout(p, const_cast<void*>(workspace), n_parts, rows, &po, &pl, &pe);
  ma.part_o = po;
  ma.part_lse = pl;
  ma.part_exp = pe;
  ma.out = out;
  ma.lse = lse;
  ma.bf16 = p->dtype == INFLLM_BF16;
  return ma;
}


infllm_status prep_append(const infllm_params* p, const infllm_memory* m, const void* q, int64_t q_head_stride,
                          const void* k, const void* v, int64_t kv_head_stride, int32_t n_q, int64_t past_len,
                          AppendArgs* a) {
  infllm_status st;
  if ((st = check_params(p)) != INFLLM_OK) return st;
  if ((st = check_store(p, m)) != INFLLM_OK) return st;
  const bool ring_used = !mean_repr(p);
  if (ring_used && m->qprefix == nullptr) return INFLLM_E_NULL;
  if (n_q < 0 || past_len < 0) return INFLLM_E_SHAPE;
  if ((k == nullptr) != (v == nullptr)) return INFLLM_E_NULL;
  if (q == nullptr) return INFLLM_E_NULL;
  if (q_head_stride < (int64_t)n_q * p->head_dim) return INFLLM_E_SHAPE;
  if (k != nullptr && ((st = check_rows(p, k, kv_head_stride, n_q)) != INFLLM_OK ||
                       (st = check_rows(p, v, kv_head_stride, n_q)) != INFLLM_OK))
    return st;
  if (ring_used && (m->ring < 1 || m->ring <= n_q)) return INFLLM_E_SHAPE;
  if (past_len + n_q > m->capacity) return INFLLM_E_RANGE;
  if (ring_used && m->rpart == nullptr) return INFLLM_E_NULL;
  if (ring_used) {
    // Partial representative scores are formed for tokens t = p - l_L (t >= l_I) of
    // the appended positions p; the running sum at t must still be in the ring
    // after this chunk's slots are written, and the key of a token inside the
    // chunk comes from k.
    const int64_t t_lo = std::max<int64_t>(p->n_init, past_len - p->n_local);
    const int64_t t_hi = past_len + n_q - p->n_local;  // exclusive
    if (t_hi > t_lo) {
      if (t_lo + m->ring < past_len + n_q) return INFLLM_E_RANGE;
      if (t_hi > past_len && k == nullptr) return INFLLM_E_NULL;
    }
  }
  a->batch = m->batch;
  a->n_q_heads = p->n_q_heads;
  a->n_kv_heads = p->n_kv_heads;
  a->head_dim = p->head_dim;
  a->n_q = n_q;
  a->ring = m->ring;
  a->n_init = p->n_init;
  a->n_local = p->n_local;
  a->past_len = past_len;
  a->capacity = m->capacity;
  a->q_head_stride = q_head_stride;
  a->kv_head_stride = kv_head_stride;
  a->q = q;
  a->k_src = k;
  a->v_src = v;
  a->k_store = m->k;
  a->v_store = m->v;
  a->qprefix = m->qprefix;
  a->rpart = m->rpart;
  a->k_rot = m->k_rot;
  a->rope = rope_args(p);
  a->var.on = 0;
  a->mean_repr = mean_repr(p);
  a->bf16 = p->dtype == INFLLM_BF16;
  return INFLLM_OK;
}

infllm_status prep_build(const infllm_params* p, const infllm_memory* m, int32_t first_unit, int32_t n_new,
                         int64_t past_len, double* repr_score, BuildArgs* a) {
  infllm_status st;
  if ((st = check_params(p)) != INFLLM_OK) return st;
  if ((st = check_store(p, m)) != INFLLM_OK) return st;
  if ((st = check_units(p, m)) != INFLLM_OK) return st;
  const bool ring_used = !mean_repr(p);
  if (ring_used && m->rpart == nullptr) return INFLLM_E_NULL;
  if (first_unit < 0 || n_new < 0 || past_len < 0 || (ring_used && m->ring < 1)) return INFLLM_E_SHAPE;
  if ((int64_t)first_unit + n_new > m->max_units) return INFLLM_E_RANGE;
  if (past_len > m->capacity) return INFLLM_E_RANGE;
  if (n_new > 0) {
    const int64_t m0 = (int64_t)p->n_init + (int64_t)first_unit * p->block_size;
    const int64_t m_last = (int64_t)p->n_init + ((int64_t)first_unit + n_new) * p->block_size - 1;
    if (m_last + p->n_local > past_len - 1) return INFLLM_E_RANGE;  // windows not appended yet: not evicted
    if (ring_used && m0 < past_len - m->ring) return INFLLM_E_RANGE;  // ring no longer holds the oldest slot
  }
  a->batch = m->batch;
  a->n_q_heads = p->n_q_heads;
  a->n_kv_heads = p->n_kv_heads;
  a->head_dim = p->head_dim;
  a->n_init = p->n_init;
  a->n_local = p->n_local;
  a->block_size = p->block_size;
  a->n_repr = p->n_repr;
  a->first_unit = first_unit;
  a->n_new = n_new;
  a->max_units = m->max_units;
  a->ring = m->ring;
  a->capacity = m->capacity;
  a->k_store = m->k;
  a->rpart = m->rpart;
  a->repr_idx = m->repr_idx;
  a->unit_ksum = m->unit_ksum;
  a->repr_score = repr_score;
  a->mean_repr = mean_repr(p);
  a->var_on = 0;
  a->bf16 = p->dtype == INFLLM_BF16;
  return INFLLM_OK;
}

infllm_status prep_score(const infllm_params* p, const infllm_memory* m, const void* q, int64_t q_head_stride,
                         int32_t n_q, int32_t n_units, float* scores, void* workspace, size_t workspace_bytes,
                         ScoreArgs* a) {
  infllm_status st;
  if ((st = check_params(p)) != INFLLM_OK) return st;
  if (m == nullptr) return INFLLM_E_NULL;
  if (m->batch < 1) return INFLLM_E_SHAPE;
  if ((st = check_units(p, m)) != INFLLM_OK) return st;
  if (n_q < 0 || n_units < 0) return INFLLM_E_SHAPE;
  if (n_units > m->max_units) return INFLLM_E_RANGE;
  a->n_units = n_units;
  a->var_on = 0;
  if (n_units == 0) return INFLLM_OK;
  if (scores == nullptr) return INFLLM_E_NULL;
  if ((st = check_rows(p, q, q_head_stride, n_q)) != INFLLM_OK) return st;
  if (workspace == nullptr) return INFLLM_E_NULL;
  if (workspace_bytes < qbar_ws_bytes(p, m->batch, n_q)) return INFLLM_E_WORKSPACE;
  if (!aligned16(workspace)) return INFLLM_E_SHAPE;
  a->batch = m->batch;
  a->n_q_heads = p->n_q_heads;
  a->n_kv_heads = p->n_kv_heads;
  a->head_dim = p->head_dim;
  a->n_q = n_q;
  a->max_units = m->max_units;
  a->q_head_stride = q_head_stride;
  a->q = q;
  a->unit_ksum = m->unit_ksum;
  a->scores = scores;
  a->qbar_parts = (float*)workspace;
  a->rope = rope_args(p);
  a->bf16 = p->dtype == INFLLM_BF16;
  return INFLLM_OK;
}

infllm_status prep_topk(int32_t rows, const float* scores, int32_t n_units, int32_t k, int32_t* idx) {
  if (rows < 0 || n_units < 0 || k < 0) return INFLLM_E_SHAPE;
  if (rows == 0 || k == 0) return INFLLM_OK;
  if (idx == nullptr) return INFLLM_E_NULL;
  if (n_units > 0 && scores == nullptr) return INFLLM_E_NULL;
  return INFLLM_OK;
}

}  // namespace

extern "C" {

const char* infllm_status_string(infllm_status s) {
  switch (s) {
    case INFLLM_OK: return "ok";
    case INFLLM_E_NULL: return "a required pointer is NULL";
    case INFLLM_E_SHAPE: return "inconsistent sizes or parameters";
    case INFLLM_E_RANGE: return "positions, units or ring slots outside the memory";
    case INFLLM_E_UNSUPPORTED: return "unsupported configuration";
    case INFLLM_E_WORKSPACE: return "workspace too small";
    case INFLLM_E_LAUNCH: return "kernel launch failed";
    case INFLLM_E_DEVICE: return "no usable gfx950 device";
  }
  return "unknown status";
}

infllm_status infllm_partition(const infllm_params* p, int64_t past_len, int64_t* n_init, int32_t* n_units,
                               int64_t* local_begin) {
  infllm_status st = check_params(p);
  if (st != INFLLM_OK) return st;
  if (n_init == nullptr || n_units == nullptr || local_begin == nullptr) return INFLLM_E_NULL;
  if (past_len < 0) return INFLLM_E_SHAPE;
  const Part r = partition(p, past_len);
  *n_init = r.n_init;
  *n_units = r.n_units;
  *local_begin = r.local_begin;
  return INFLLM_OK;
}

// Bytes of the per-tile unit-mass partials infllm_step_mass keeps at the end of
// the workspace (0 where the attention cannot write them: units not made of
// whole 64-key tiles).
static size_t mass_part_bytes(const infllm_params* p, int32_t batch, int32_t n_q) {
  if (p->topk <= 0 || p->block_size % 64 != 0 || p->n_init % 64 != 0 || n_q <= 0) return 0;
  const int G = p->n_q_heads / p->n_kv_heads;
  return (size_t)batch * p->n_kv_heads * p->topk * (p->block_size / 64) * (size_t)G * n_q * sizeof(float2);
}

size_t infllm_workspace_bytes(const infllm_params* p, int32_t batch, int32_t n_q) {
  if (check_params(p) != INFLLM_OK || batch < 1 || n_q < 0) return 0;
  const int G = p->n_q_heads / p->n_kv_heads;
  int parts = attend_max_parts(p->dtype == INFLLM_BF16, G, n_q, max_virtual_keys(p, n_q));
  if (remap(p)) parts = std::max(parts, 2);
  size_t a = attend_ws_bytes(p, batch, n_q, parts);
  size_t b = qbar_ws_bytes(p, batch, n_q);
  size_t r = a > b ? a : b;
  r = (r + 255) & ~(size_t)255;
  return r + ((mass_part_bytes(p, batch, n_q) + 255) & ~(size_t)255);
}

size_t infllm_attend_workspace_bytes(const infllm_params* p, int32_t batch, int32_t n_q) {
  return infllm_workspace_bytes(p, batch, n_q);
}

infllm_status infllm_append(const infllm_params* p, const infllm_memory* m, const void* q, int64_t q_head_stride,
                            const void* k, const void* v, int64_t kv_head_stride, int32_t n_q, int64_t past_len,
                            void* stream) {
  AppendArgs a;
  infllm_status st = prep_append(p, m, q, q_head_stride, k, v, kv_head_stride, n_q, past_len, &a);
  if (st != INFLLM_OK) return st;
  if ((st = check_device()) != INFLLM_OK) return st;
  return launch_status(launch_append(a, (hipStream_t)stream, nullptr, nullptr));
}

infllm_status infllm_build_units(const infllm_params* p, const infllm_memory* m, int32_t first_unit, int32_t n_new,
                                 int64_t past_len, double* repr_score, void* stream) {
  BuildArgs a;
  infllm_status st = prep_build(p, m, first_unit, n_new, past_len, repr_score, &a);
  if (st != INFLLM_OK || n_new == 0) return st;
  if ((st = check_device()) != INFLLM_OK) return st;
  return launch_status(launch_build_units(a, (hipStream_t)stream));
}

infllm_status infllm_score_units(const infllm_params* p, const infllm_memory* m, const void* q, int64_t q_head_stride,
                                 int32_t n_q, int32_t n_units, float* scores, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  ScoreArgs a;
  infllm_status st = prep_score(p, m, q, q_head_stride, n_q, n_units, scores, workspace, workspace_bytes, &a);
  if (st != INFLLM_OK || n_units == 0) return st;
  if ((st = check_device()) != INFLLM_OK) return st;
  return launch_status(launch_score(a, (hipStream_t)stream));
}

infllm_status infllm_select_topk(int32_t rows, const float* scores, int32_t n_units, int32_t k, int32_t* idx,
                                 void* stream) {
  infllm_status st = prep_topk(rows, scores, n_units, k, idx);
  if (st != INFLLM_OK || rows == 0 || k == 0) return st;
  if ((st = check_device()) != INFLLM_OK) return st;
  return launch_status(launch_select_topk(rows, scores, n_units, k, idx, (hipStream_t)stream));
}

infllm_status infllm_attend_partial(const infllm_params* p, const infllm_memory* m, const void* q,
                                    int64_t q_head_stride, int32_t n_q, int64_t past_len, const int32_t* idx,
                                    int32_t k, void* out, int64_t out_head_stride, float* lse, void* workspace,
                                    size_t workspace_bytes, int32_t* n_parts, void* stream) {
  if (n_parts == nullptr) return INFLLM_E_NULL;
  AttendArgs a;
  infllm_status st = prepare_attend(p, m, q, q_head_stride, n_q, past_len, idx, k, out, out_head_stride, lse,
                                    workspace, workspace_bytes, &a);
  if (st != INFLLM_OK) return st;
  *n_parts = a.parts;
  if (n_q == 0) return INFLLM_OK;
  if ((st = check_device()) != INFLLM_OK) return st;
  return launch_status(launch_attend(a, (hipStream_t)stream));
}

infllm_status infllm_lse_merge(const infllm_params* p, int32_t batch, int32_t n_q, int32_t n_parts,
                               const void* workspace, size_t workspace_bytes, void* out, int64_t out_head_stride,
                               float* lse, void* stream) {
  infllm_status st;
  if ((st = check_params(p)) != INFLLM_OK) return st;
  if (batch < 1 || n_q < 0 || n_parts < 2) return INFLLM_E_SHAPE;
  if (workspace == nullptr) return INFLLM_E_NULL;
  if (workspace_bytes < attend_ws_bytes(p, batch, n_q, n_parts)) return INFLLM_E_WORKSPACE;
  if ((st = check_rows(p, out, out_head_stride, n_q)) != INFLLM_OK) return st;
  if (n_q == 0) return INFLLM_OK;
  if ((st = check_device()) != INFLLM_OK) return st;
  MergeArgs ma = merge_args(p, batch, n_q, n_parts, workspace, out, out_head_stride, lse);
  return launch_status(launch_merge(ma, (hipStream_t)stream));
}

infllm_status infllm_chunk_attend(const infllm_params* p, const infllm_memory* m, const void* q, int64_t q_head_stride,
                                  int32_t n_q, int64_t past_len, const int32_t* idx, int32_t k, void* out,
                                  int64_t out_head_stride, float* lse, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  AttendArgs a;
  infllm_status st = prepare_attend(p, m, q, q_head_stride, n_q, past_len, idx, k, out, out_head_stride, lse,
                                    workspace, workspace_bytes, &a);
  if (st != INFLLM_OK) return st;
  if (n_q == 0) return INFLLM_OK;
  if ((st = check_device()) != INFLLM_OK) return st;
  if ((st = launch_status(launch_attend(a, (hipStream_t)stream))) != INFLLM_OK) return st;
  if (a.parts == 1) return INFLLM_OK;
  MergeArgs ma = merge_args(p, m->batch, n_q, a.parts, workspace, out, out_head_stride, lse);
  return launch_status(launch_merge(ma, (hipStream_t)stream));
}

infllm_status infllm_chunk_attend_noalloc(const infllm_params* p, const infllm_memory* m, const void* q,
                                          int64_t q_head_stride, int32_t n_q, int64_t past_len, const int32_t* idx,
                                          int32_t k, void* out, int64_t out_head_stride, float* lse, void* stream) {
  // the scratch array's address on this device (looked up once per device), then
  // the workspace path of infllm_chunk_attend with the array as the workspace
  infllm_status st;
  if ((st = check_device()) != INFLLM_OK) return st;
  void* ws = scratch_device_ptr();
  if (ws == nullptr) return INFLLM_E_DEVICE;
  AttendArgs a;
  if ((st = prepare_attend(p, m, q, q_head_stride, n_q, past_len, idx, k, out, out_head_stride, lse, ws,
                           kScratchBytes, &a)) != INFLLM_OK)
    return st;
  if (n_q == 0) return INFLLM_OK;
  if ((st = launch_status(launch_attend(a, (hipStream_t)stream))) != INFLLM_OK) return st;
  if (a.parts == 1) return INFLLM_OK;
  MergeArgs ma = merge_args(p, m->batch, n_q, a.parts, ws, out, out_head_stride, lse);
  return launch_status(launch_merge(ma, (hipStream_t)stream));
}

// Validation and arguments of the unit-mass launch (infllm_unit_mass, and the
// fallback of infllm_step_mass).  *skip: nothing to launch.
static infllm_status prep_unit_mass(const infllm_params* p, const infllm_memory* m, const void* q,
                                    int64_t q_head_stride, int32_t n_q, int64_t past_len, const int32_t* idx,
                                    int32_t k, const float* lse, float decay, float* mass, float* freq, MassArgs* a,
                                    bool* skip) {
  infllm_status st;
  *skip = false;
  if ((st = check_params(p)) != INFLLM_OK) return st;
  if ((st = check_store(p, m)) != INFLLM_OK) return st;
  if (n_q < 0 || past_len < 0 || k < 0) return INFLLM_E_SHAPE;
  if (!std::isfinite(decay) || decay < 0.f) return INFLLM_E_SHAPE;
  if (past_len + n_q > m->capacity) return INFLLM_E_RANGE;
  if (k > kMassMaxK) return INFLLM_E_UNSUPPORTED;
  if (p->dtype == INFLLM_BF16 && (uint64_t)m->capacity * (uint64_t)p->head_dim * 2u > 0xFFFFFFFFull)
    return INFLLM_E_UNSUPPORTED;
  const Part part = partition(p, past_len);
  if (freq != nullptr && part.n_units > m->max_units) return INFLLM_E_RANGE;
  if (k > 0) {
    if (idx == nullptr || mass == nullptr) return INFLLM_E_NULL;
    if (n_q > 0) {
      if (lse == nullptr) return INFLLM_E_NULL;
      if ((st = check_rows(p, q, q_head_stride, n_q)) != INFLLM_OK) return st;
    }
  }
  if (k == 0 && (freq == nullptr || part.n_units == 0)) {
    *skip = true;
    return INFLLM_OK;
  }
  std::memset(a, 0, sizeof(*a));
  a->rows = m->batch * p->n_kv_heads;
  a->n_q_heads = p->n_q_heads;
  a->n_kv_heads = p->n_kv_heads;
  a->head_dim = p->head_dim;
  a->n_q = n_q;
  a->k = k;
  a->n_units = part.n_units;
  a->max_units = m->max_units;
  a->block_size = p->block_size;
  a->n_init = p->n_init;
  a->capacity = m->capacity;
  a->q_head_stride = q_head_stride;
  a->sm_scale = p->sm_scale;
  a->decay = decay;
  a->q = q;
  a->k_store = m->k;
  a->idx = idx;
  a->lse = lse;
  a->mass = mass;
  a->freq = part.n_units > 0 ? freq : nullptr;
  a->rope = rope_args(p);
  a->bf16 = p->dtype == INFLLM_BF16;
  return INFLLM_OK;
}

infllm_status infllm_unit_mass(const infllm_params* p, const infllm_memory* m, const void* q,
                               int64_t q_head_stride, int32_t n_q, int64_t past_len, const int32_t* idx, int32_t k,
                               const float* lse, float decay, float* mass, float* freq, void* stream) {
  MassArgs a;
  bool skip;
  infllm_status st = prep_unit_mass(p, m, q, q_head_stride, n_q, past_len, idx, k, lse, decay, mass, freq, &a,
                                    &skip);
  if (st != INFLLM_OK || skip) return st;
  if ((st = check_device()) != INFLLM_OK) return st;
  return launch_status(launch_unit_mass(a, (hipStream_t)stream));
}

struct MassRequest {
  float decay;
  float* mass;
  float* freq;
};

static infllm_status step_impl(const infllm_params* p, const infllm_memory* m, const void* q,
                               int64_t q_head_stride, const void* k, const void* v, int64_t kv_head_stride,
                               int32_t n_q, int64_t past_len, int32_t units_built, float* scores, int32_t* idx,
                               void* out, int64_t out_head_stride, float* lse, void* workspace,
                               size_t workspace_bytes, void* stream, const MassRequest* mr) {
  infllm_status st;
  if ((st = check_params(p)) != INFLLM_OK) return st;
  if (m == nullptr) return INFLLM_E_NULL;
  if (past_len < 0 || units_built < 0) return INFLLM_E_SHAPE;
  const Part part = partition(p, past_len);
  if (units_built > part.n_units) return INFLLM_E_SHAPE;
  BuildArgs ba;
  AppendArgs aa;
  ScoreArgs sa;
  AttendArgs at;
  MassArgs mass_args;
  bool mass_skip = true;
  char* mass_area = nullptr;
  if (mr != nullptr) {
    // the unit mass of this step's lookup, validated like infllm_unit_mass
    if ((st = prep_unit_mass(p, m, q, q_head_stride, n_q, past_len, idx, p->topk, lse, mr->decay, mr->mass, mr->freq,
                             &mass_args, &mass_skip)) != INFLLM_OK)
      return st;
    // the attention's per-tile partials at the end of the workspace, when it has room
    const size_t mb = mass_part_bytes(p, m->batch, n_q);
    if (mb > 0 && workspace != nullptr && workspace_bytes >= mb + 256) {
      const size_t off = (workspace_bytes - mb) & ~(size_t)255;
      mass_area = (char*)workspace + off;
      workspace_bytes = off;
    }
  }
  if ((st = prep_build(p, m, units_built, part.n_units - units_built, past_len, nullptr, &ba)) != INFLLM_OK) return st;
  if ((st = prep_append(p, m, q, q_head_stride, k, v, kv_head_stride, n_q, past_len, &aa)) != INFLLM_OK) return st;
  if ((st = prep_score(p, m, q, q_head_stride, n_q, part.n_units, scores, workspace, workspace_bytes, &sa)) !=
      INFLLM_OK)
    return st;
  const int32_t rows = m->batch * p->n_kv_heads;
  if ((st = prep_topk(rows, scores, part.n_units, p->topk, idx)) != INFLLM_OK) return st;
  if ((st = prepare_attend(p, m, q, q_head_stride, n_q, past_len, idx, p->topk, out, out_head_stride, lse, workspace,
                           workspace_bytes, &at)) != INFLLM_OK)
    return st;
  if ((st = check_device()) != INFLLM_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  // Unit construction reads ring slots of positions >= its first token m0; the
  // append writes the slots of [past_len, past_len + n_q).  When the ring is
  // large enough for those never to coincide, both run in one launch.
  // (The mean representation reads only keys already in the store: always one launch.)
  const int64_t m0 = (int64_t)p->n_init + (int64_t)units_built * p->block_size;
  const bool mean = mean_repr(p);
  const bool fuse = ba.n_new > 0 && n_q > 0 && (mean || m0 >= past_len + n_q - m->ring);
  if (ba.n_new > 0 && !fuse && (st = launch_status(launch_build_units(ba, s))) != INFLLM_OK) return st;
  // The append also yields the chunk's group-query sums, which scoring consumes
  // directly: the scan total, or with the mean representation (no scan) the
  // partial sums of its query-sum blocks.
  float* qbar = (float*)workspace;
  const int qbar_parts = mean ? score_qbar_parts(p->n_q_heads / p->n_kv_heads, n_q) : 1;
  if ((st = launch_status(launch_append(aa, s, part.n_units > 0 ? qbar : nullptr, fuse ? &ba : nullptr))) !=
      INFLLM_OK)
    return st;
  if (part.n_units > 0) {
    sa.qbar_parts = qbar;
    if (n_q == 0) {
      if ((st = launch_status(launch_score(sa, s))) != INFLLM_OK) return st;
    } else if ((st = launch_status(launch_score_given_qbar(sa, qbar_parts, s))) != INFLLM_OK) {
      return st;
    }
  }
  // The matrix-core attention selects the units itself (one launch fewer on the
  // step's critical path) when the score rows are short enough for its prologue;
  // otherwise the selection kernel runs first.  With no units yet the selection
  // kernel still writes the -1 padding of idx.
  const bool select_in_attend = p->topk > 0 && p->topk <= kFusedSelectMaxK && part.n_units > 0 &&
                                part.n_units <= kFusedSelectMax && attend_uses_mfma(at);
  if (select_in_attend) {
    at.sel_scores = scores;
    at.sel_stride = part.n_units;
    at.sel_units = part.n_units;
    at.idx_out = idx;
  } else if (p->topk > 0 &&
             (st = launch_status(launch_select_topk(rows, scores, part.n_units, p->topk, idx, s))) != INFLLM_OK) {
    return st;
  }
  // With the unit mass asked for and the lookup inside the attention, the
  // attention also writes each unit tile's per-row sums of P; one small launch
  // after the merge turns them into the masses (else the unit-mass kernel).
  const bool mass_in_attend = mr != nullptr && !mass_skip && select_in_attend && mass_area != nullptr;
  if (mass_in_attend) {
    at.mass_part = (float2*)mass_area;
    at.mass_tiles = p->topk * (p->block_size / 64);
  }
  if (n_q > 0) {
    if ((st = launch_status(launch_attend(at, s))) != INFLLM_OK) return st;
    if (at.parts > 1) {
      MergeArgs ma = merge_args(p, m->batch, n_q, at.parts, workspace, out, out_head_stride, lse);
      if ((st = launch_status(launch_merge(ma, s))) != INFLLM_OK) return st;
    }
  }
  if (mr == nullptr || mass_skip) return INFLLM_OK;
  if (!mass_in_attend) return launch_status(launch_unit_mass(mass_args, s));
  MassPartsArgs mp;
  std::memset(&mp, 0, sizeof(mp));
  mp.rows = rows;
  mp.n_q_heads = p->n_q_heads;
  mp.n_kv_heads = p->n_kv_heads;
  mp.n_q = n_q;
  mp.k = p->topk;
  mp.n_sel = at.geom.n_sel;
  mp.n_units = part.n_units;
  mp.max_units = m->max_units;
  mp.tiles_per_unit = p->block_size / 64;
  mp.mass_tiles = at.mass_tiles;
  mp.decay = mr->decay;
  mp.mass_part = at.mass_part;
  mp.idx = idx;
  mp.lse = lse;
  mp.mass = mr->mass;
  mp.freq = mass_args.freq;
  return launch_status(launch_unit_mass_parts(mp, s));
}

infllm_status infllm_step(const infllm_params* p, const infllm_memory* m, const void* q, int64_t q_head_stride,
                          const void* k, const void* v, int64_t kv_head_stride, int32_t n_q, int64_t past_len,
                          int32_t units_built, float* scores, int32_t* idx, void* out, int64_t out_head_stride,
                          float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  return step_impl(p, m, q, q_head_stride, k, v, kv_head_stride, n_q, past_len, units_built, scores, idx, out,
                   out_head_stride, lse, workspace, workspace_bytes, stream, nullptr);
}

infllm_status infllm_step_mass(const infllm_params* p, const infllm_memory* m, const void* q,
                               int64_t q_head_stride, const void* k, const void* v, int64_t kv_head_stride,
                               int32_t n_q, int64_t past_len, int32_t units_built, float* scores, int32_t* idx,
                               void* out, int64_t out_head_stride, float* lse, float decay, float* mass, float* freq,
                               void* workspace, size_t workspace_bytes, void* stream) {
  const MassRequest mr = {decay, mass, freq};
  return step_impl(p, m, q, q_head_stride, k, v, kv_head_stride, n_q, past_len, units_built, scores, idx, out,
                   out_head_stride, lse, workspace, workspace_bytes, stream, &mr);
}

infllm_status infllm_step_varlen(const infllm_params* p, const infllm_memory* m, const void* q,
                                 int64_t q_head_stride, const void* k, const void* v, int64_t kv_head_stride,
                                 int32_t n_q, const int64_t* past_lens, const int32_t* units_built, float* scores,
                                 int32_t* idx, void* out, int64_t out_head_stride, float* lse, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  infllm_status st;
  if ((st = check_params(p)) != INFLLM_OK) return st;
  if (m == nullptr || past_lens == nullptr || units_built == nullptr) return INFLLM_E_NULL;
  if (m->batch < 1) return INFLLM_E_SHAPE;
  if (m->batch > kMaxVarBatch) return INFLLM_E_UNSUPPORTED;
  const int B = m->batch;
  const bool mean = mean_repr(p);
  // Every sequence's stages are validated as a step of its own; the launches
  // then carry all sequences, each kernel deriving a sequence's geometry from
  // its past length.  The first sequence's arguments supply the shared fields.
  BuildArgs ba;
  AppendArgs aa;
  ScoreArgs sa;
  std::memset(&sa, 0, sizeof(sa));
  AttendArgs at;
  int32_t n_units[kMaxVarBatch];
  int n_units_max = 0, new_max = 0, parts = 1, n_sel_max = 0, nv_max = 0;
  bool fuse = n_q > 0;
  for (int b = 0; b < B; ++b) {
    const int64_t past = past_lens[b];
    if (past < 0 || units_built[b] < 0) return INFLLM_E_SHAPE;
    const Part part = partition(p, past);
    if (units_built[b] > part.n_units) return INFLLM_E_SHAPE;
    BuildArgs bb;
    AppendArgs ab;
    ScoreArgs sb;
    AttendArgs tb;
    if ((st = prep_build(p, m, units_built[b], part.n_units - units_built[b], past, nullptr, &bb)) != INFLLM_OK)
      return st;
    if ((st = prep_append(p, m, q, q_head_stride, k, v, kv_head_stride, n_q, past, &ab)) != INFLLM_OK) return st;
    if ((st = prep_score(p, m, q, q_head_stride, n_q, part.n_units, scores, workspace, workspace_bytes, &sb)) !=
        INFLLM_OK)
      return st;
    if ((st = prepare_attend(p, m, q, q_head_stride, n_q, past, idx, p->topk, out, out_head_stride, lse, workspace,
                             workspace_bytes, &tb)) != INFLLM_OK)
      return st;
    if (b == 0) {
      ba = bb;
      aa = ab;
      at = tb;
    }
    // (scoring arguments are complete only where the sequence has units)
    if (part.n_units > 0 && n_units_max == 0) sa = sb;
    n_units[b] = part.n_units;
    n_units_max = std::max(n_units_max, part.n_units);
    new_max = std::max(new_max, bb.n_new);
    parts = std::max(parts, tb.parts);
    n_sel_max = std::max(n_sel_max, tb.geom.n_sel);
    nv_max = std::max(nv_max, tb.geom.n_virtual);
    const int64_t m0 = (int64_t)p->n_init + (int64_t)units_built[b] * p->block_size;
    if (bb.n_new > 0 && !mean && m0 < past + n_q - m->ring) fuse = false;
    ba.var_first[b] = units_built[b];
    ba.var_count[b] = bb.n_new;
    aa.var.past[b] = past;
    at.var.past[b] = past;
  }
  const int32_t rows = B * p->n_kv_heads;
  if (p->topk > 0 && idx == nullptr) return INFLLM_E_NULL;
  if (n_units_max > 0 && scores == nullptr) return INFLLM_E_NULL;
  // every sequence's parts fit the workspace (each was checked for its own count)
  ba.var_on = 1;
  ba.n_new = new_max;
  aa.var.on = 1;
  sa.var_on = 1;
  sa.n_units = n_units_max;
  for (int b = 0; b < B; ++b) sa.var_units[b] = n_units[b];
  sa.score_stride = m->max_units;
  at.var.on = 1;
  at.parts = parts;
  at.geom.n_sel = n_sel_max;  // bounds only: each kernel derives its sequence's values
  at.geom.n_virtual = nv_max;
  partial_layout(p, workspace, parts, (int64_t)B * p->n_q_heads * n_q, &at.part_o, &at.part_lse, &at.part_exp);
  if ((st = check_device()) != INFLLM_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if (new_max > 0 && !fuse && (st = launch_status(launch_build_units(ba, s))) != INFLLM_OK) return st;
  float* qbar = (float*)workspace;
  const int qbar_parts = mean ? score_qbar_parts(p->n_q_heads / p->n_kv_heads, n_q) : 1;
  if ((st = launch_status(launch_append(aa, s, n_units_max > 0 ? qbar : nullptr,
                                        (fuse && new_max > 0) ? &ba : nullptr))) != INFLLM_OK)
    return st;
  if (n_units_max > 0) {
    sa.qbar_parts = qbar;
    if (n_q == 0) {
      if ((st = launch_status(launch_score(sa, s))) != INFLLM_OK) return st;
    } else if ((st = launch_status(launch_score_given_qbar(sa, qbar_parts, s))) != INFLLM_OK) {
      return st;
    }
  }
  // As in infllm_step: the attention selects each sequence's units itself when
  // every score row is short enough (a sequence without units gets -1 padding).
  if (p->topk > 0 && p->topk <= kFusedSelectMaxK && n_units_max > 0 && n_units_max <= kFusedSelectMax &&
      attend_uses_mfma(at)) {
    at.sel_scores = scores;
    at.sel_stride = m->max_units;
    at.sel_units = n_units_max;
    at.idx_out = idx;
  } else if (p->topk > 0) {
    TopkRows tr;
    tr.rows_per_seq = p->n_kv_heads;
    for (int b = 0; b < B; ++b) tr.row_n[b] = n_units[b];
    if ((st = launch_status(launch_select_topk_var(rows, scores, m->max_units, n_units_max, tr, p->topk, idx, s))) !=
        INFLLM_OK)
      return st;
  }
  if (n_q == 0) return INFLLM_OK;
  if ((st = launch_status(launch_attend(at, s))) != INFLLM_OK) return st;
  if (at.parts == 1) return INFLLM_OK;
  MergeArgs ma = merge_args(p, B, n_q, at.parts, workspace, out, out_head_stride, lse);
  return launch_status(launch_merge(ma, s));
}

}  // extern "C"
