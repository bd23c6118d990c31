// Chunk attention over Concat(I, selected units, L, X) (Section 3.1) in bf16 on
// CDNA4 matrix cores (v_mfma_f32_32x32x16_bf16), fp32 accumulation.
//
// Work decomposition
//   rows   : per (sequence, kv head) the G*n_q query rows (row r -> query i = r/G,
//            head g*G + r%G), so the G heads sharing a K/V tile are packed together;
//            256 rows per workgroup (one per compute unit), 32 per wave, so each
//            K/V tile crosses into LDS once for all 8 waves.
//   keys   : the virtual key axis (see StepGeom) in tiles of 64 keys, gathered
//            straight from the token-ordered store (a selected unit is contiguous)
//            into LDS by direct global->LDS loads (no staging registers) through
//            three buffers; optionally split into parts whose partial softmaxes
//            are merged afterwards by log-sum-exp.
// Per wave and key tile:
//   S^T = K Q^T  : A = K tile rows from LDS, B = the wave's Q rows held in VGPRs.
//                  The 32x32 accumulator gives each lane one query row and 16 keys.
//   online softmax in the exp2 domain, row max combined across the two lane halves.
//   O^T += V^T P^T: B = P^T taken directly from the S^T accumulator (no shuffle);
//                  A = V^T fragments read from the key-major V tile with the LDS
//                  transpose read (ds_read_b64_tr_b16), in the key order the
//                  accumulator layout gives P^T.
#include "launch.h"
#include "topk_select.h"

namespace infllm {
namespace {

constexpr int KB = 64;      // keys per tile
constexpr int NWAVE = 8;
constexpr int ROWS_WG = 32 * NWAVE;
static_assert(ROWS_WG == kMfmaRowsPerWg, "row tiling shared with the part chooser");

typedef short i16x4 __attribute__((ext_vector_type(4)));
#define INFLLM_LDS __attribute__((address_space(3)))

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Direct global->LDS loads (16 bytes per lane; lane i lands at LDS byte
// lds + 16*i, lds taken from M0).  Written as inline assembly so that the
// compiler does not guard every later LDS read with a wait for these loads: the
// kernel waits for them itself (s_waitcnt before the barrier that publishes a
// tile).  No compiler-generated code in these kernels uses M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// Contiguous run: wave-uniform base address plus a per-lane 32-bit byte offset.
__device__ __forceinline__ void lds_load_run(uint32_t lds, const void* base, uint32_t off) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" : : "s"(lds), "v"(off), "s"(base) : "m0");
}
// Gather: a full per-lane address.
__device__ __forceinline__ void lds_load_lane(uint32_t lds, const void* p) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" : : "s"(lds), "v"(p) : "m0");
}
#pragma clang diagnostic pop

// Values the compiler must treat as produced here (keeps derived addresses from
// being hoisted out of the tile loop into long-lived registers).
__device__ __forceinline__ uint32_t opaque_v(uint32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}
__device__ __forceinline__ uint32_t opaque_s(uint32_t x) {
  asm volatile("" : "+s"(x));
  return x;
}

// Both LDS tiles are key-major [64 keys][D], unpadded, with the 16-byte granules
// of row r XOR-swizzled (granule g stored at g ^ swz(r)), and a 1 KB direct-load
// instruction still writes one contiguous LDS range.  gfx950 LDS serves 256
// bytes per clock (64 banks); for D = 128 (256-byte rows) the 4-bit swizzle
// below makes both fragment reads conflict-free: the K reads (16 consecutive
// rows, one granule each, per clock) and the transposed V reads (per 32 lanes:
// 4 consecutive rows x 64 bytes).  For D = 64 the 3-bit swizzle r & 7.
template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return r & 7;
}
template <int D>
__device__ __forceinline__ int tile_off(int r, int g) { return r * D + 8 * (g ^ swz<D>(r)); }

constexpr int NBUF = 3;         // K and V tile buffers
constexpr int kMaskCost = 6;  // cost of a masked tile, in quarters of a plain tile (measured ~1.5x)
constexpr int kSelTiles4 = 5;  // the in-prologue unit selection, in quarters of a plain tile
constexpr int kSelTiles4Long = 16;  // the same for rows of more than kFusedSelectShort units
constexpr int kRunTable = 1024;  // run starts kept in LDS for the part's tiles
constexpr int kSelLds = 1024;    // lookup entries kept in LDS
static_assert(kFusedSelectMaxK <= kSelLds, "a selected lookup row fits in LDS");

template <int D>
struct Smem {
  bf16_t k[NBUF][KB * D];
  bf16_t v[NBUF][KB * D];
  int64_t runs[kRunTable];  // run start of tile t_begin + i (see tile_run_start)
  int32_t sidx[kSelLds];    // the lookup row (its first kSelLds entries)
  uint8_t kvalid[NBUF][KB];
};

// Publish LDS tiles to the workgroup: wait until at most N of this wave's
// direct loads are still in flight (older loads -- the tiles about to be read
// -- have landed in LDS) and its own LDS traffic is done, then barrier.  Written
// out so that no wait for the younger loads is implied.
template <int N>
__device__ __forceinline__ void publish_barrier() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N));
  // LDS-only fences: order this wave's LDS accesses around the barrier without
  // a wait for its outstanding global loads.
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// SEL > 0: the workgroups select the lookup themselves from a.sel_scores, SEL
// keys of a score row per thread (2: rows of at most kFusedSelectShort units;
// 16: longer rows, filtered first) -- kernels of their own, so that the plain
// kernel's code is unaffected.  MASS (with SEL):
// for every tile of the looked-up units the kernel also stores, per query row,
// the tile's sum of P = exp2(S*c2 - m) and the running max m it was formed
// against, from which the attention mass of each unit follows once the final
// lse is known (mass_parts_kernel).
template <int D, int SEL, bool MASS>
__global__ void __launch_bounds__(64 * NWAVE, 1) attend_mfma_kernel(AttendArgs a) {
  constexpr int CH = D / 8;                   // 16-byte granules per row
  constexpr int KSTEPS = D / 16;              // MFMA k-steps over the head dim
  constexpr int DBLK = D / 32;                // 32-wide output blocks
  constexpr int RPI = 64 / CH;                // tile rows per 1 KB load instruction
  constexpr int NI = KB * D * 2 / (NWAVE * 1024);  // load instructions per wave per tile (K or V)
  static_assert(NI * NWAVE * RPI == KB, "tile rows covered exactly once");
  static_assert(2 * NI <= KSTEPS, "one load per chunk of the MFMA phase");
  __shared__ __attribute__((aligned(256))) Smem<D> sm;

  const int G = a.n_q_heads / a.n_kv_heads;
  const int R = G * a.geom.n_q;
  const int n_row_tiles = (R + ROWS_WG - 1) / ROWS_WG;
  // XCD-aware order, reversed so that the workgroups dispatched first are those
  // with the most work: the last key part (it holds the causal diagonal of X) and
  // the last row tiles (their queries see the most of X)
  const int L = (int)gridDim.x - 1 - xcd_logical_block(blockIdx.x, gridDim.x);
  const int rt = L % n_row_tiles;
  const int tmp = L / n_row_tiles;
  const int part = tmp % a.parts;
  const int bg = tmp / a.parts;
  const int b = bg / a.n_kv_heads, g = bg - b * a.n_kv_heads;
  // this sequence's step (its own past length in a variable-length batch)
  const SeqStep sq = seq_step(a, b);
  const StepGeom& geo = sq.geom;
  const int mem_len = sq.mem_len, parts_mem = sq.parts_mem;

  // This part's tiles.  Without the positional remap the parts split the tiles
  // evenly.  With it, parts [0, parts_mem) split the memory tiles [0,
  // ceil(mem_len/KB)) (I and the units: unrotated keys, queries turned by R(l_L))
  // and the other parts the local tiles [floor(mem_len/KB), n_tiles) (L and X:
  // rotated keys, queries at their own positions); a tile holding keys of both
  // kinds is taken by both sides, each masking the other's keys.
  const int n_tiles = (geo.n_virtual + KB - 1) / KB;
  const bool remap = a.rope.on != 0;
  const bool mem_part = part < parts_mem;
  int rt0 = 0, rt1 = n_tiles, rpart = part, rparts = a.parts;
  if (mem_part) {
    rt1 = (mem_len + KB - 1) / KB;
    rparts = parts_mem;
  } else if (parts_mem > 0) {
    rt0 = mem_len / KB;
    rpart = part - parts_mem;
    rparts = a.parts - parts_mem;
  }
  // The parts split the range by cost rather than by tile count: a tile holding
  // current-token keys (the causal diagonal, masked) costs kMaskCost/4 of a plain
  // tile, so the part that takes the diagonal takes fewer tiles and all parts end
  // together.
  const int v_x0 = geo.n_virtual - geo.n_q;  // first current-token key
  auto part_bound = [&](int pp) -> int {  // first tile of part pp of rparts
    const int a_x = min(max(v_x0 / KB, rt0), rt1);
    if constexpr (!SEL) {
      const int64_t c_plain = 4LL * (a_x - rt0);
      const int64_t c_all = c_plain + (int64_t)kMaskCost * (rt1 - a_x);
      const int64_t c = c_all * pp / rparts;
      if (c <= c_plain) return rt0 + (int)((c + 3) / 4);
      return a_x + (int)((c - c_plain + kMaskCost - 1) / kMaskCost);
    }
    // The parts that read unit keys also select the units (see below), about
    // kSelTiles tiles of work each.  The tiles up to the end of the units are
    // charged that work spread over them, for the share of the parts expected to
    // fall there (costs in 1/64 of a plain tile).
    const int u_end = (geo.n_init + geo.n_sel * geo.block_size + KB - 1) / KB;
    const int s_end = min(max(u_end, rt0), a_x);
    constexpr int64_t kPlain = 64, kMask = 16 * kMaskCost;
    constexpr int64_t kSel4 = SEL > 2 ? kSelTiles4Long : kSelTiles4;
    const int64_t kSel = kPlain + (kPlain * kSel4 * rparts) / (4 * max(1, rt1 - rt0));
    const int64_t c_sel = kSel * (s_end - rt0);
    const int64_t c_plain = c_sel + kPlain * (a_x - s_end);
    const int64_t c_all = c_plain + kMask * (rt1 - a_x);
    const int64_t c = c_all * pp / rparts;
    if (c <= c_sel) return rt0 + (int)((c + kSel - 1) / kSel);
    if (c <= c_plain) return s_end + (int)((c - c_sel + kPlain - 1) / kPlain);
    return a_x + (int)((c - c_plain + kMask - 1) / kMask);
  };
  const int t_begin = part_bound(rpart);
  int t_end = part_bound(rpart + 1);
  {
    const int i_max = (min(R, (rt + 1) * ROWS_WG) - 1) / G;
    t_end = min(t_end, (v_x0 + i_max) / KB + 1);  // tiles past this are fully causal-masked
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, gsel = lane >> 5;
  const int row = rt * ROWS_WG + wave * 32 + n;
  const bool row_ok = row < R;
  const int qi = row_ok ? row / G : 0;
  // last virtual key this row may see: causal within X (which also excludes the
  // ragged end), or for a memory part of the remap the last memory key
  const int vlim = mem_part ? mem_len - 1 : v_x0 + qi;
  const int qh = g * G + (row_ok ? row - qi * G : 0);

  const int32_t* idx_row = a.idx + (int64_t)bg * geo.idx_stride;
  const bf16_t* kbase = (const bf16_t*)(remap && !mem_part ? a.k_rot : a.k_store) + (int64_t)bg * a.capacity * D;
  const bf16_t* vbase = (const bf16_t*)a.v_store + (int64_t)bg * a.capacity * D;

  // The lookup row goes to LDS (run starts then read LDS, not global memory) in
  // the same round trip as the Q rows; one barrier publishes it together with
  // the check for skipped (out-of-range) entries, which send every tile through
  // the per-key gather path and the validity mask.
  bool bad = false;
  if constexpr (!SEL) {
    for (int u = tid; u < geo.n_sel; u += 64 * NWAVE) {
      const int x = idx_row[u];
      if (u < kSelLds) sm.sidx[u] = x;
      bad |= (x < 0 || x >= geo.n_units);
    }
  }
  // Lookup inside the attention: a workgroup selects the units itself when a
  // tile it reads (its own, the run-start table's and the loads issued ahead:
  // [t_begin, t_end + 4)) holds unit keys; the workgroup of row tile 0 and part
  // 0 always does, and writes the row out.  Every entry is then valid.  The
  // score row is loaded here, its latency overlapping the Q loads below.
  static_assert(SEL == 0 || SEL == 2 || SEL == tk::kMaxPer, "select keys per thread");
  static_assert(tk::kThreads == 64 * NWAVE && 2 * tk::kThreads >= kFusedSelectShort &&
                    tk::kMaxPer * tk::kThreads >= kFusedSelectMax,
                "select layout");
  const bool sel_writer = SEL > 0 && rt == 0 && part == 0;
  bool sel_here = sel_writer;
  if constexpr (SEL) {
    const int u_t0 = geo.n_init / KB, u_t1 = (geo.n_init + geo.n_sel * geo.block_size + KB - 1) / KB;
    sel_here |= t_begin < u_t1 && t_end + 4 > u_t0;
  }
  const bool sel_all = geo.n_sel == 0 || geo.n_sel == geo.n_units;  // every unit (or none) is looked up
  constexpr int SK = SEL > 0 ? SEL : 1;
  uint32_t skey[SK] = {};
  if (SEL > 0 && sel_here && !sel_all) {
    const float* srow = a.sel_scores + (int64_t)bg * a.sel_stride;
#pragma unroll
    for (int j = 0; j < SK; ++j) skey[j] = tk::order_key(srow[min(tid + j * tk::kThreads, geo.n_units - 1)]);
  }
  // Q rows of this wave as the B operand (8 bf16 per lane per k-step).
  bf16x8 qreg[KSTEPS];
  {
    const bf16_t* qp = (const bf16_t*)a.q + (int64_t)(b * a.n_q_heads + qh) * a.q_head_stride + (int64_t)qi * D;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      u32x4 raw = row_ok ? *(const u32x4*)(qp + 16 * s + 8 * gsel) : u32x4{0, 0, 0, 0};
      if (remap) {
        // memory parts: the query turned by R(l_L); local parts: at its own position
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int pr = 8 * s + 4 * gsel + j;  // the pair held in word j
          float cs, sn;
          if (mem_part) {
            cs = a.rope.mem_cos[pr];
            sn = a.rope.mem_sin[pr];
          } else {
            rope_cos_sin(a.rope, geo.past_len + qi, pr, cs, sn);
          }
          const float x0 = __uint_as_float(raw[j] << 16), x1 = __uint_as_float(raw[j] & 0xFFFF0000u);
          raw[j] = (uint32_t)f32_to_bf16(x0 * cs - x1 * sn) | ((uint32_t)f32_to_bf16(x0 * sn + x1 * cs) << 16);
        }
      }
      qreg[s] = __builtin_bit_cast(bf16x8, raw);
    }
  }
  if (SEL > 0 && sel_here) {
    if (sel_all) {
      for (int u = tid; u < geo.n_sel; u += 64 * NWAVE) sm.sidx[u] = u;
    } else {
      auto valid = [&](int j) { return tid + j * tk::kThreads < geo.n_units; };
      auto index = [&](int j) { return tid + j * tk::kThreads; };
      uint32_t thr;
      int rem;
      bool ge;
      // long rows: the filter first (it declines, uniformly, when the bound it
      // finds leaves more than a thread's worth of candidates)
      bool done = false;
      if constexpr (SEL > 2) done = geo.n_sel <= tk::kThreads && tk::filtered_select<SK>(skey, geo.n_units, geo.n_sel, sm.sidx);
      if (!done) {
        tk::radix_threshold<SK>(skey, valid, geo.n_sel, thr, rem, ge);
        tk::write_selection<SK>(skey, valid, index, thr, rem, ge, geo.n_sel, sm.sidx);
      }
    }
    __syncthreads();
    if (sel_writer) {
      int32_t* orow = a.idx_out + (int64_t)bg * geo.idx_stride;
      for (int u = tid; u < geo.idx_stride; u += 64 * NWAVE) orow[u] = u < geo.n_sel ? sm.sidx[u] : -1;
    }
  }
  const bool has_invalid = __syncthreads_or(bad) != 0;

  // Direct loads: instruction j of wave w fills LDS granules [(NI*w + j)*64, +64)
  // of the tile, lane l writing granule slot l; that slot belongs to tile row
  // r_j = (NI*w + j)*RPI + l / CH and holds its global granule (l % CH) ^ swz(r_j).
  // Under the swizzle r_j = r_0 + RPI*j and granule_j = granule_0 ^ XJ*j.
  constexpr int XJ = D == 128 ? 1 : 0;
  const int lrow0 = NI * wave * RPI + lane / CH;
  const int lgran0 = (lane % CH) ^ swz<D>(lrow0);

  // A tile inside one segment (I, one selected unit, or the L+X run) maps to 64
  // consecutive store positions: the common case, gathered with no per-key work.
  // Returns that first position (uniform across the workgroup) or -1.
  auto tile_run_start = [&](int tile) -> int64_t {
    const int v0 = tile * KB;
    if (has_invalid || v0 + KB > geo.n_virtual) return -1;
    if (v0 + KB <= geo.n_init) return v0;
    if (v0 < geo.n_init) return -1;
    const int w = v0 - geo.n_init;
    const int sel_len = geo.n_sel * geo.block_size;
    if (w >= sel_len) return geo.local_begin + (w - sel_len);
    if (w + KB > sel_len) return -1;
    const int u = w / geo.block_size;
    if ((w + KB - 1) / geo.block_size != u) return -1;
    const int bu = u < kSelLds ? sm.sidx[u] : idx_row[u];
    return (int64_t)geo.unit_base + (int64_t)bu * geo.block_size + (w - u * geo.block_size);
  };
  // Store position of virtual key v (-1: skipped unit entry), with the lookup
  // entry read from LDS: on the per-key path of tiles that span several runs a
  // global read would wait behind the tile loads in flight.
  auto vpos = [&](int v) -> int64_t {
    if (v < geo.n_init) return v;
    const int w = v - geo.n_init;
    const int sel_len = geo.n_sel * geo.block_size;
    if (w >= sel_len) return geo.local_begin + (w - sel_len);
    const int u = w / geo.block_size;
    const int bu = u < kSelLds ? sm.sidx[u] : idx_row[u];
    if (bu < 0 || bu >= geo.n_units) return -1;
    return (int64_t)geo.unit_base + (int64_t)bu * geo.block_size + (w - u * geo.block_size);
  };
  auto uniform64 = [](int64_t x) -> int64_t {
    return ((int64_t)__builtin_amdgcn_readfirstlane((int)(x >> 32)) << 32) |
           (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
  };

  // Byte offsets of this wave's 1 KB slices in the LDS tiles, and the per-lane
  // byte offset of the granule each lane fetches within a contiguous run.
  const uint32_t lds_k0 = (uint32_t)(uintptr_t)(INFLLM_LDS bf16_t*)sm.k[0];
  const uint32_t lds_v0 = (uint32_t)(uintptr_t)(INFLLM_LDS bf16_t*)sm.v[0];
  const uint32_t lds_k = lds_k0 + NI * wave * 1024;
  const uint32_t lds_v = lds_v0 + NI * wave * 1024;
  constexpr uint32_t kTileBytes = KB * D * 2;
  // byte offset of instruction j's granule within a contiguous run:
  // (run_off0 ^ 16*XJ*j) + 1024*j
  const uint32_t run_off0 = (uint32_t)(lrow0 * D + 8 * lgran0) * 2u;

  // Direct loads of tile `tile` (run start `run0`) into buffer `buf` of K or of
  // V.  A key that is not part of the context (ragged end, skipped unit entry)
  // reads position 0 -- always written -- and is masked to -inf before the
  // softmax (the ragged end by the causal bound, a skipped entry by kvalid, which
  // the K load records), so its K/V never contribute.
  auto issue = [&](int tile, int64_t run0, int buf, auto is_k) {
    constexpr bool IS_K = decltype(is_k)::value;
    const uint32_t ld = (IS_K ? lds_k : lds_v) + buf * kTileBytes;
    const bf16_t* base = IS_K ? kbase : vbase;
    if (run0 >= 0) {
      const bf16_t* src = base + run0 * D;
      const uint32_t ro = opaque_v(run_off0);
#pragma unroll
      for (int j = 0; j < NI; ++j) lds_load_run(ld + j * 1024, src + 512 * j, ro ^ (16u * XJ * j));
    } else {
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int r = lrow0 + RPI * j;
        const int v = tile * KB + r;
        int64_t pos = v < geo.n_virtual ? vpos(v) : -1;
        if (IS_K && lane % CH == 0) sm.kvalid[buf][r] = pos >= 0;
        pos = pos >= 0 ? pos : 0;
        lds_load_lane(ld + j * 1024, base + pos * D + 8 * (lgran0 ^ (XJ * j)));
      }
    }
  };
  // The same loads split in two: per-lane byte offsets from the store base
  // (formed at the top of an iteration; per-key gather on the uncommon path) and
  // the loads themselves, issued one per chunk of the MFMA phase so that the
  // waves of the workgroup do not queue a burst of them after the barrier.  The
  // host guarantees that one (sequence, kv head) slice of the store spans less
  // than 4 GiB, so the offsets fit 32 bits.
  auto load_offsets = [&](int tile, int64_t run0, int buf, bool is_k, uint32_t (&off)[NI]) {
    if (run0 >= 0) {
      const uint32_t ro = opaque_v(run_off0) + (uint32_t)run0 * (2u * D);
#pragma unroll
      for (int j = 0; j < NI; ++j) off[j] = (ro ^ (16u * XJ * j)) + 1024u * j;
    } else {
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int r = lrow0 + RPI * j;
        const int v = tile * KB + r;
        int64_t pos = v < geo.n_virtual ? vpos(v) : -1;
        if (is_k && lane % CH == 0) sm.kvalid[buf][r] = pos >= 0;
        pos = pos >= 0 ? pos : 0;
        off[j] = (uint32_t)pos * (2u * D) + 16u * (lgran0 ^ (XJ * j));
      }
    }
  };

  // Loop-invariant per-lane LDS offsets (elements); the swizzle depends on the
  // row only through r & 15, so +16 and +32 rows keep it.
  //  K fragment (S^T A operand) of k-step s: lane (n, gsel) reads row n (+32 for
  //  the second key block), granule 2s + gsel.
  //  V^T fragment (O^T A operand) of output block db: a transposed read by lane
  //  (h = lane/16, q = (lane%16)/4, m = lane%4) addresses key row
  //  16*j + 4*(h/2) + 8*e + q and dims 32*db + 16*(h%2) + 4*m .. +4; each lane then
  //  holds dim 32*db + lane%32 of keys 16*j + 4*gsel + 8*e + 0..3 -- the key order
  //  of the P^T operand taken from the S^T accumulator.
  // Under the swizzle these offsets are XOR-related (buffers start at multiples
  // of 256 bytes, so the XOR commutes with adding the buffer address):
  //   K, k-step s          : koff0 ^ 32*s                         (bytes)
  //   V^T, block db, half e: (voff0 ^ 64*db ^ VX*e) + e*16*D      (bytes)
  // so only two bases stay in registers and each tile derives its addresses.
  constexpr uint32_t VX = D == 128 ? 32 : 0;
  const uint32_t koff0 = 2u * tile_off<D>(n, gsel);
  uint32_t voff0;
  {
    const int h = lane >> 4, q = (lane & 15) >> 2, m = lane & 3;
    const int vr = 4 * (h >> 1) + q, d0 = 16 * (h & 1) + 4 * m;
    voff0 = 2u * (tile_off<D>(vr, d0 >> 3) + (d0 & 7));
  }
  auto kfrag_at = [&](uint32_t kaddr, int kb, int s) {
    return *(const INFLLM_LDS bf16x8*)(uintptr_t)((kaddr ^ (32u * s)) + kb * 64u * D);
  };
  auto vfrag_at = [&](uint32_t vaddr, int db, int j) {
    const uint32_t a0 = (vaddr ^ (64u * db)) + j * 32u * D;
    const uint32_t a1 = ((vaddr ^ (64u * db) ^ VX) + 16u * D) + j * 32u * D;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((INFLLM_LDS i16x4*)(uintptr_t)a0);
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((INFLLM_LDS i16x4*)(uintptr_t)a1);
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };
  // per-tile fragment base addresses (the buffer address is made opaque so that
  // the derived addresses are formed per tile instead of held in registers)
  auto kaddr_of = [&](int kbuf) { return opaque_s(lds_k0 + kbuf * kTileBytes) + koff0; };
  auto vaddr_of = [&](int vbuf) { return opaque_s(lds_v0 + vbuf * kTileBytes) + voff0; };

  f32x16 oacc[DBLK];
#pragma unroll
  for (int db = 0; db < DBLK; ++db)
#pragma unroll
    for (int j = 0; j < 16; ++j) oacc[db][j] = 0.f;
  float m_run = -__builtin_inff();
  float l_run = 0.f;
  const float c2 = a.sm_scale * 1.4426950408889634f;

  // ---- the pieces of one tile's work ----------------------------------------
  // S^T = K Q^T for the tile in K buffer `kb`: two accumulator chains (keys
  // [0,32) and [32,64)), K fragments read one k-step ahead.
  auto qk = [&](int kbuf, f32x16 (&sacc)[2]) {
    const uint32_t ka = kaddr_of(kbuf);
    auto kfrag = [&](int kb, int s) { return kfrag_at(ka, kb, s); };
    bf16x8 a0[2], a1[2];
    a0[0] = kfrag(0, 0);
    a1[0] = kfrag(1, 0);
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      if (s + 1 < KSTEPS) {
        a0[(s + 1) & 1] = kfrag(0, s + 1);
        a1[(s + 1) & 1] = kfrag(1, s + 1);
      }
      if (s == 0) {
        const f32x16 zero = {};
        sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[0], qreg[0], zero, 0, 0, 0);
        sacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[0], qreg[0], zero, 0, 0, 0);
      } else {
        sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[s & 1], qreg[s], sacc[0], 0, 0, 0);
        sacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[s & 1], qreg[s], sacc[1], 0, 0, 0);
      }
    }
  };
  // Mask of tile t: key kl is visible to query qi iff its virtual index is at
  // most vlim and, with skipped unit entries present, its kvalid flag (K buffer
  // kbuf) is set.
  auto apply_mask = [&](int t, int kbuf, f32x16 (&sacc)[2]) {
    const int lim = vlim - t * KB - 4 * gsel;
    uint32_t kv[4][2];
    if (has_invalid) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j4 = 0; j4 < 4; ++j4)
          kv[j4][kb] = *(const uint32_t*)&sm.kvalid[kbuf][32 * kb + 8 * j4 + 4 * gsel];
    }
    // one uniform branch for the tile, none per element
    if (has_invalid) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int c = 32 * kb + 8 * (j >> 2) + (j & 3);
          const bool vis = c <= lim && ((kv[j >> 2][kb] >> (8 * (j & 3))) & 0xFFu) != 0;
          sacc[kb][j] = vis ? sacc[kb][j] : -__builtin_inff();
        }
    } else {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int c = 32 * kb + 8 * (j >> 2) + (j & 3);
          sacc[kb][j] = c <= lim ? sacc[kb][j] : -__builtin_inff();
        }
    }
  };
  // Row max of the tile in the exp2 domain (both lane halves combined).
  auto tile_max = [&](const f32x16 (&sacc)[2]) {
    float mx = -__builtin_inff();
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 16; ++j) mx = fmaxf(mx, sacc[kb][j]);
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
    return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * c2;  // c2 > 0
  };
  // Lazy running max.  P is formed against the running max m_run without first
  // taking the tile's own maximum; a row whose half-tile sum of P exceeds kLazy
  // (2^16: P stays far inside the float and bf16 range) has met keys well above
  // m_run, and only then is the tile's maximum taken and the row rescaled (a rare
  // path; the decision is wave-uniform, and both lane halves of a row share
  // m_run).  While a row has seen no visible key (m_run = -inf) any nonzero P
  // takes that path, so the first visible tile sets m_run.
  constexpr float kLazy = 65536.f;
  auto lazy_bound = [&]() { return m_run == -__builtin_inff() ? 0.f : kLazy; };
  auto force_max = [&](float mx) {
    const float m_new = fmaxf(m_run, mx);
    const float alpha = (m_new == -__builtin_inff()) ? 1.f : fast_exp2(m_run - m_new);
    l_run *= alpha;
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) oacc[db][j] *= alpha;
    m_run = m_new;
  };
  // Tile t's contribution to the unit masses (MASS): for a tile of the looked-up
  // units (whole tiles: l_I and l_bs are multiples of the tile), the row's sum of
  // P over the tile's 64 keys (this lane's half plus the other lane half's) and
  // the running max it was formed against.  Later rescales of l_run leave the
  // stored pair valid: it carries its own max.
  auto mass_tile = [&](int t, float half_sum) {
    const int ut = t - geo.n_init / KB;  // tile index within the units
    const int n_ut = geo.n_sel * (geo.block_size / KB);
    if (ut < 0 || ut >= n_ut) return;
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(half_sum), __float_as_uint(half_sum), false,
                                                      false);
    const float tsum = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
    if (row_ok && gsel == 0)
      a.mass_part[((int64_t)bg * a.mass_tiles + ut) * R + row] = make_float2(tsum, m_run);
  };
  // Two P values as a bf16 pair (one v_cvt_pk_bf16_f32), added unrounded to the
  // two running row sums (the normaliser keeps float32 precision; rounding only
  // the PV operand moves O by at most 2^-9 relative).
  auto p_pair = [&](float z0, float z1, float nm, float (&acc)[2]) -> uint32_t {
    const float e0 = fast_exp2(__builtin_fmaf(z0, c2, nm));
    const float e1 = fast_exp2(__builtin_fmaf(z1, c2, nm));
    acc[0] += e0;
    acc[1] += e1;
    bf16x2 pr;
    pr[0] = (__bf16)e0;
    pr[1] = (__bf16)e1;
    return __builtin_bit_cast(uint32_t, pr);
  };
  // One 16-key half of P = exp2(S*c2 - m_run) as the bf16 operand pair, and its row sum.
  auto half_p = [&](const f32x16& sh, u32x4 (&ph)[2]) {
    const float nm = (m_run == -__builtin_inff()) ? 0.f : -m_run;
    float ps[2] = {0.f, 0.f};
#pragma unroll
    for (int w = 0; w < 8; ++w) ph[w >> 2][w & 3] = p_pair(sh[2 * w], sh[2 * w + 1], nm, ps);
    return ps[0] + ps[1];
  };
  auto as_bf16x8 = [](const u32x4& w) { return __builtin_bit_cast(bf16x8, w); };
  // O^T += V^T P^T over the four 16-key steps (V buffer vbuf); DBLK independent
  // accumulator chains, each V^T fragment two transposed 8-byte reads.
  auto pv = [&](int vbuf, const bf16x8 (&pb)[2][2]) {
    const uint32_t vaddr = vaddr_of(vbuf);
    auto vfrag = [&](int db, int j) { return vfrag_at(vaddr, db, j); };
    bf16x8 va[DBLK];
#pragma unroll
    for (int db = 0; db < DBLK; ++db) va[db] = vfrag(db, 0);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int db = 0; db < DBLK; ++db) {
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[db], pb[j >> 1][j & 1], oacc[db], 0, 0, 0);
        if (j + 1 < 4) va[db] = vfrag(db, j + 1);
      }
    }
  };

  // ---- software pipeline over the part's tiles ---------------------------------
  // Tile x lives in K buffer and V buffer (x - t_begin) % 3.  Iteration t runs
  // PV(t) and QK(t+1): the matrix cores work on QK(t+1) while the vector ALUs
  // form the keys [32, 64) half of P(t), and on PV(t) while they take the mask
  // and max of tile t+1 and form the keys [0, 32) half of P(t+1) with the
  // running max (redone in the rare iteration whose tile raises the max past the
  // lazy-rescale threshold), which balances the vector work over both phases.  Loads are
  // issued two iterations ahead, K three tiles ahead and V two tiles ahead, so
  // each buffer is refilled only after the barrier that retires its last readers:
  //   top of iteration t: wait for K(t+1), V(t) (issued two iterations ago; the
  //   2*NI loads of the previous iteration may stay in flight), barrier; issue
  //   K(t+3) into the K buffer of tile t (QK(t) ran in iteration t-1) and V(t+2)
  //   into the V buffer of tile t-1.
  // Every iteration issues exactly 2*NI loads per wave, which keeps the wait
  // count constant: a tile past the part's end is simply loaded too (a tile past
  // the key axis reads position 0), into a buffer nobody reads.  Run starts are
  // looked up at the end of an iteration, so their scalar loads complete under
  // the barrier.
  // Tiles wholly before X need no mask unless skipped unit entries exist.
  const int t_plain = has_invalid ? t_begin : max(t_begin, min(t_end, (mem_part ? mem_len : v_x0) / KB));
  int64_t run_k = -1, run_v = -1;  // run starts of the next K and V loads: tiles t+3, t+2
  // Run starts of the part's tiles, computed once by all lanes into LDS; the
  // per-iteration lookup is then an LDS read (a global read here would wait
  // behind the tile loads in flight).  Tiles past the table compute directly.
  const int n_table = min(kRunTable, t_end + 4 - t_begin);
  for (int i = tid; i < n_table; i += 64 * NWAVE) sm.runs[i] = tile_run_start(t_begin + i);
  // early half of a lookup: the LDS read (or -2 when the tile is past the table)
  auto run_read = [&](int tile) -> int64_t {
    const int i = tile - t_begin;
    return i < n_table ? sm.runs[i] : -2;
  };
  auto run_finish = [&](int tile, int64_t r) -> int64_t { return uniform64(r != -2 ? r : tile_run_start(tile)); };
  f32x16 sA[2], sB[2];
  // p0: the keys [0, 32) half of P(t), formed in the previous iteration's phase 2
  // (or the prologue), and l_pend its row sum, added to l_run once the other half
  // of the tile has passed its lazy-max check; replaced here by that half of P(t+1).
  u32x4 p0[2];
  float l_pend = 0.f;
  auto iteration = [&](int t, f32x16 (&cur)[2], f32x16 (&nxt)[2], auto mask_next) {
    const int bc = (t - t_begin) % NBUF;
    const int bn = bc == NBUF - 1 ? 0 : bc + 1, bp = bc == 0 ? NBUF - 1 : bc - 1;
    publish_barrier<2 * NI>();
    uint32_t off_k[NI], off_v[NI];
    load_offsets(t + 3, run_k, bc, true, off_k);
    load_offsets(t + 2, run_v, bp, false, off_v);
    const uint32_t ld_k = lds_k + bc * kTileBytes, ld_v = lds_v + bp * kTileBytes;
    const int64_t run_next = run_read(t + 4);  // consumed after phase 2

    // Phases 1 and 2 run at raised wave priority (s_setprio 1), the barrier,
    // address and bookkeeping at normal priority: a wave in its MFMA phases
    // wins the issue slots of its SIMD over a wave doing bookkeeping (measured a
    // few percent faster than uniform priority).
    __builtin_amdgcn_s_setprio(1);
    // Phase 1: QK(t+1) on the matrix cores, the keys [32, 64) half of P(t) on the
    // vector ALUs.  Chunk s issues the K fragment reads of k-step s+1, the two
    // MFMAs of k-step s and EPC elements of that half of P(t); scheduling fences
    // keep that interleave.
    float neg_m = (m_run == -__builtin_inff()) ? 0.f : -m_run;
    u32x4 w1[2];
    float ps1[2] = {0.f, 0.f};  // two partial row sums (shorter dependency chains)
    {
      const uint32_t ka = kaddr_of(bn);
      auto kfrag = [&](int kb, int s) { return kfrag_at(ka, kb, s); };
      bf16x8 a0[2], a1[2];
      a0[0] = kfrag(0, 0);
      a1[0] = kfrag(1, 0);
      constexpr int EPC = 16 / KSTEPS;  // elements of P(t)'s keys [32, 64) half per chunk
      static_assert(EPC % 2 == 0, "P elements are formed in bf16 pairs");
#pragma unroll
      for (int s = 0; s < KSTEPS; ++s) {
        if (s + 1 < KSTEPS) {
          a0[(s + 1) & 1] = kfrag(0, s + 1);
          a1[(s + 1) & 1] = kfrag(1, s + 1);
        }
        if (s == 0) {
          const f32x16 zero = {};
          nxt[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[0], qreg[0], zero, 0, 0, 0);
          nxt[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[0], qreg[0], zero, 0, 0, 0);
        } else {
          nxt[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[s & 1], qreg[s], nxt[0], 0, 0, 0);
          nxt[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[s & 1], qreg[s], nxt[1], 0, 0, 0);
        }
        // the s-th of this wave's 2*NI loads of K(t+3) and V(t+2)
        if (s < NI) lds_load_run(ld_k + s * 1024, kbase, off_k[s]);
        else if (s < 2 * NI) lds_load_run(ld_v + (s - NI) * 1024, vbase, off_v[s - NI]);
#pragma unroll
        for (int i = 0; i < EPC; i += 2) {
          const int w = (EPC * s + i) >> 1;  // bf16 pair index within the half
          w1[w >> 2][w & 3] = p_pair(cur[1][2 * w], cur[1][2 * w + 1], neg_m, ps1);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    float psum1 = ps1[0] + ps1[1];
    // lazy-max check of that half before it reaches the matrix cores: on the rare
    // row that exceeds the bound, rescale to the tile's maximum and redo both halves
    if (__ballot(psum1 > lazy_bound())) {
      force_max(tile_max(cur));
      l_pend = half_p(cur[0], p0);
      psum1 = half_p(cur[1], w1);
      neg_m = (m_run == -__builtin_inff()) ? 0.f : -m_run;
    }
    l_run += l_pend + psum1;
    if constexpr (MASS) mass_tile(t, l_pend + psum1);

    // Phase 2: PV(t) on the matrix cores; on the vector ALUs the mask of tile t+1
    // (one 8-element group of its 32 accumulator elements per step) and, four
    // elements per step, the keys [0, 32) half of P(t+1) against the running max
    // (checked after the phase).
    u32x4 q0[2];
    float ps0[2] = {0.f, 0.f};
    {
      constexpr bool MASK = decltype(mask_next)::value;
      const uint32_t vaddr = vaddr_of(bc);
      auto vfrag = [&](int db, int j) { return vfrag_at(vaddr, db, j); };
      const int lim = vlim - (t + 1) * KB - 4 * gsel;  // mask bound of tile t+1
      uint32_t kv[4][2];
      if (MASK && has_invalid) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int j4 = 0; j4 < 4; ++j4)
            kv[j4][kb] = *(const uint32_t*)&sm.kvalid[bn][32 * kb + 8 * j4 + 4 * gsel];
      }
      bf16x8 va[DBLK];
#pragma unroll
      for (int db = 0; db < DBLK; ++db) va[db] = vfrag(db, 0);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int db = 0; db < DBLK; ++db) {
          oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[db], as_bf16x8(j < 2 ? p0[j & 1] : w1[j & 1]),
                                                            oacc[db], 0, 0, 0);
          if (j + 1 < 4) va[db] = vfrag(db, j + 1);
        }
        if constexpr (MASK) {
          // 8 of the 32 scores of tile t+1: elements [8j, 8j+8); one uniform branch
          // per step, none per element
          if (has_invalid) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              const int e = 8 * j + i, kb = e >> 4, jj = e & 15;
              const int c = 32 * kb + 8 * (jj >> 2) + (jj & 3);
              const bool vis = c <= lim && ((kv[jj >> 2][kb] >> (8 * (jj & 3))) & 0xFFu) != 0;
              nxt[kb][jj] = vis ? nxt[kb][jj] : -__builtin_inff();
            }
          } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              const int e = 8 * j + i, kb = e >> 4, jj = e & 15;
              const int c = 32 * kb + 8 * (jj >> 2) + (jj & 3);
              nxt[kb][jj] = c <= lim ? nxt[kb][jj] : -__builtin_inff();
            }
          }
        }
        // P(t+1), keys [0, 32): elements [4j, 4j+4) (masked by step j/2 <= j)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          const int w = 2 * j + i;
          q0[w >> 2][w & 3] = p_pair(nxt[0][2 * w], nxt[0][2 * w + 1], neg_m, ps0);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __builtin_amdgcn_s_setprio(0);
    p0[0] = q0[0];
    p0[1] = q0[1];
    l_pend = ps0[0] + ps0[1];
    if (__ballot(l_pend > lazy_bound())) {
      force_max(tile_max(nxt));
      l_pend = half_p(nxt[0], p0);
    }
    run_v = run_k;
    run_k = run_finish(t + 4, run_next);
  };
  auto copy_state = [](f32x16 (&dst)[2], const f32x16 (&src)[2]) {
    dst[0] = src[0];
    dst[1] = src[1];
  };

  if (t_begin < t_end) {
    // K(t0), V(t0), K(t0+1) | V(t0+1), K(t0+2): the last two groups play the
    // loads of "the previous iteration" for the first iteration's wait.
    const int64_t r0 = uniform64(tile_run_start(t_begin));
    const int64_t r1 = uniform64(tile_run_start(t_begin + 1));
    const int64_t r2 = uniform64(tile_run_start(t_begin + 2));
    issue(t_begin, r0, 0, std::true_type{});
    issue(t_begin, r0, 0, std::false_type{});
    issue(t_begin + 1, r1, 1, std::true_type{});
    issue(t_begin + 1, r1, 1, std::false_type{});
    issue(t_begin + 2, r2, 2, std::true_type{});
    run_v = r2;
    run_k = uniform64(tile_run_start(t_begin + 3));
    publish_barrier<4 * NI>();  // K(t0) has landed
    qk(0, sA);
    if (t_begin >= t_plain) apply_mask(t_begin, 0, sA);
    if (!mem_part && parts_mem > 0 && t_begin * KB < mem_len) {
      // the first local tile also holds the last memory keys: hide them here
      const int lo = mem_len - t_begin * KB - 4 * gsel;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j)
          if (32 * kb + 8 * (j >> 2) + (j & 3) < lo) sA[kb][j] = -__builtin_inff();
    }
    force_max(tile_max(sA));  // the first tile sets the running max
    l_pend = half_p(sA[0], p0);

    int t = t_begin;
    // next tile unmasked
    for (; t + 2 < t_plain; t += 2) {
      iteration(t, sA, sB, std::false_type{});
      iteration(t + 1, sB, sA, std::false_type{});
    }
    if (t + 1 < t_plain) {
      iteration(t, sA, sB, std::false_type{});
      copy_state(sA, sB);
      ++t;
    }
    // next tile masked
    for (; t + 2 < t_end; t += 2) {
      iteration(t, sA, sB, std::true_type{});
      iteration(t + 1, sB, sA, std::true_type{});
    }
    if (t + 1 < t_end) {
      iteration(t, sA, sB, std::true_type{});
      copy_state(sA, sB);
      ++t;
    }
    // drain: P and PV of the last tile (then no load is left in flight)
    publish_barrier<0>();
    u32x4 w1[2];
    float psum1 = half_p(sA[1], w1);
    if (__ballot(psum1 > lazy_bound())) {
      force_max(tile_max(sA));
      l_pend = half_p(sA[0], p0);
      psum1 = half_p(sA[1], w1);
    }
    l_run += l_pend + psum1;
    if constexpr (MASS) mass_tile(t, l_pend + psum1);
    const bf16x8 pb[2][2] = {{as_bf16x8(p0[0]), as_bf16x8(p0[1])}, {as_bf16x8(w1[0]), as_bf16x8(w1[1])}};
    pv((t - t_begin) % NBUF, pb);
  }

  // Epilogue: combine the two lane halves' partial sums; write O (bf16, one part)
  // or the scaled fp16 partial row and lse.  The accumulator layout gives each
  // lane 8-byte pieces of its row; they are staged through LDS (the tile buffers
  // are free once every wave has passed the barrier below) so that each store
  // moves 16 contiguous bytes and a wave's store covers four whole rows.
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_v = (m_run == -__builtin_inff() || l_tot <= 0.f)
                          ? -__builtin_inff()
                          : (m_run + __log2f(l_tot)) * 0.6931471805599453f;
  const bool one_part = a.parts == 1;
  float sc = inv;
  int ex = 0;
  if (!one_part) {
    // fp16 partial row scaled by 2^-e (both lane halves of the row agree on e)
    float amax = 0.f;
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) amax = fmaxf(amax, fabsf(oacc[db][j]));
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(amax), __float_as_uint(amax), false, false);
    amax = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1])) * inv;
    ex = partial_row_exponent(amax);
    sc = inv * exp2_int(-ex);
  }
  constexpr int kRowBytes = D * 2;
  constexpr int kStageRow = kRowBytes + 16;  // padded: the 32 rows of a wave spread over the LDS banks
  static_assert(NWAVE * 32 * kStageRow <= (int)sizeof(sm.k) + (int)sizeof(sm.v), "staging fits the tile buffers");
  __syncthreads();  // every wave is done with the tile buffers
  {
    INFLLM_LDS char* stage = (INFLLM_LDS char*)(INFLLM_LDS bf16_t*)sm.k[0] + wave * 32 * kStageRow;
#pragma unroll
    for (int db = 0; db < DBLK; ++db) {
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int d = 32 * db + 8 * jq + 4 * gsel;
        const float o0 = oacc[db][4 * jq] * sc, o1 = oacc[db][4 * jq + 1] * sc;
        const float o2 = oacc[db][4 * jq + 2] * sc, o3 = oacc[db][4 * jq + 3] * sc;
        u32x2 w;
        if (one_part) {
          w[0] = (uint32_t)f32_to_bf16(o0) | ((uint32_t)f32_to_bf16(o1) << 16);
          w[1] = (uint32_t)f32_to_bf16(o2) | ((uint32_t)f32_to_bf16(o3) << 16);
        } else {
          w[0] = pack_f16x2(o0, o1);
          w[1] = pack_f16x2(o2, o3);
        }
        *(INFLLM_LDS u32x2*)(stage + n * kStageRow + d * 2) = w;
      }
    }
  }
  if (row_ok && gsel == 0) {
    const int64_t grow = ((int64_t)(b * a.n_q_heads + qh)) * geo.n_q + qi;
    if (one_part) {
      if (a.lse != nullptr) a.lse[grow] = lse_v;
    } else {
      const int64_t rows_total = (int64_t)a.batch * a.n_q_heads * geo.n_q;
      a.part_lse[(int64_t)part * rows_total + grow] = lse_v;
      a.part_exp[(int64_t)part * rows_total + grow] = ex;
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
  {
    constexpr int CPR = kRowBytes / 16;  // 16-byte chunks per row
    const INFLLM_LDS char* stage = (const INFLLM_LDS char*)(const INFLLM_LDS bf16_t*)sm.k[0] + wave * 32 * kStageRow;
    const int64_t rows_total = (int64_t)a.batch * a.n_q_heads * geo.n_q;
#pragma unroll
    for (int k = 0; k < 32 * CPR / 64; ++k) {
      const int c = 64 * k + lane, r = c / CPR, ch = c % CPR;
      const int row = rt * ROWS_WG + wave * 32 + r;
      if (row >= R) continue;
      const u32x4 w = *(const INFLLM_LDS u32x4*)(stage + r * kStageRow + ch * 16);
      const int ri = row / G, rh = g * G + (row - ri * G);
      char* dst;
      if (one_part)
        dst = (char*)a.out + ((int64_t)(b * a.n_q_heads + rh) * a.out_head_stride + (int64_t)ri * D) * 2;
      else
        dst = (char*)a.part_o + ((int64_t)part * rows_total + (int64_t)(b * a.n_q_heads + rh) * geo.n_q + ri) * kRowBytes;
      *(u32x4*)(dst + ch * 16) = w;
    }
  }
}

}  // namespace

hipError_t launch_attend_mfma(const AttendArgs& a, hipStream_t s) {
  const int G = a.n_q_heads / a.n_kv_heads;
  const int R = G * a.geom.n_q;
  const int n_row_tiles = (R + ROWS_WG - 1) / ROWS_WG;
  const int blocks = n_row_tiles * a.parts * a.batch * a.n_kv_heads;
  const dim3 grid(blocks), block(64 * NWAVE);
  const bool sel = a.sel_scores != nullptr, mass = sel && a.mass_part != nullptr;
  if (sel && (a.sel_units < 1 || a.sel_units > kFusedSelectMax)) return hipErrorInvalidValue;
  const bool long_rows = sel && a.sel_units > kFusedSelectShort;
#define INFLLM_ATTEND_MFMA(DD)                                                                         \
  do {                                                                                                 \
    if (mass && long_rows) hipLaunchKernelGGL((attend_mfma_kernel<DD, 16, true>), grid, block, 0, s, a); \
    else if (mass) hipLaunchKernelGGL((attend_mfma_kernel<DD, 2, true>), grid, block, 0, s, a);          \
    else if (long_rows) hipLaunchKernelGGL((attend_mfma_kernel<DD, 16, false>), grid, block, 0, s, a);   \
    else if (sel) hipLaunchKernelGGL((attend_mfma_kernel<DD, 2, false>), grid, block, 0, s, a);          \
    else hipLaunchKernelGGL((attend_mfma_kernel<DD, 0, false>), grid, block, 0, s, a);                   \
  } while (0)
  if (a.head_dim == 128) INFLLM_ATTEND_MFMA(128);
  else INFLLM_ATTEND_MFMA(64);
#undef INFLLM_ATTEND_MFMA
  return hipGetLastError();
}

}  // namespace infllm
