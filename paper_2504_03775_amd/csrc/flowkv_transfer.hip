// Segment-coalesced KV-cache copy for gfx950 (MI355X).
//
// FlowKV (arXiv 2504.03775), section 3.3: after bidirectional segment
// alignment every aligned run of blocks is moved by one operation, and Eq. 5's
// block-major layout (B, L, 2, H) makes a block's K and V of every layer one
// contiguous range.  Here the whole plan -- every run, every layer, K and V --
// is one kernel launch on one device; the unit of work is a tile of
// `unroll` lines, a line being one 16-byte vector per thread of a workgroup.
//
// Work decomposition.  A plan covers total_blocks logical blocks; block g's
// bytes are split into tiles_per_block tiles, giving
// units = total_blocks * tiles_per_block tiles, walked grid-stride (by
// default one tile per workgroup).  By default the blocks are visited in a
// fixed scattered order (x -> x * m mod total_blocks), so the workgroups
// resident at one moment spread over the whole plan instead of streaming
// one window of neighbouring tiles; between two block-major pools the
// tiles go tile-major (tile 0 of every block in that order, then tile 1, and
// so on).  A workgroup finds the run holding
// its tile by a galloping search over the runs' `first` fields, starting
// where equal-length runs would put it: O(log distance) per jump, nothing
// while it stays inside a run.
//
// Addressing.  Within a block, byte offset o belongs to chunk r = o / H
// (layer r / 2, K for even r, V for odd r) at offset o % H.  Block-major
// pools address base + b * BB + o; layer-major pools address
// layer_base[l] + (kv * B + b) * H + o % H.  When H is a multiple of the line
// (the usual case, H = 4 KiB or 32 KiB for Llama shapes), every line lies in
// one chunk and all address arithmetic is wave-uniform: each load is a scalar
// base plus the lane's 16-byte offset.  Other H use per-lane division by H
// (Granlund-Montgomery multiply-shift) and the layer tables staged in LDS.
//
// The data is never interpreted: the copy is byte-exact for any dtype.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>

#include "flowkv.h"
#include "flowkv_status.h"

using flowkv::fail;
using flowkv::ok;

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct PoolArg {
  char* base[FLOWKV_MAX_LAYERS];
  int64_t num_blocks;
};

// Plans of up to kInlineRuns records can travel inside the kernel arguments.
constexpr int kInlineRuns = FLOWKV_INLINE_RUNS;

// The launch's geometry and plan size, common to both argument forms.
struct XferShape {
  const flowkv_segment* segs;
  int64_t chunk_bytes;      // H (bytes of one block/layer/K-or-V slab)
  int64_t block_bytes;      // BB = 2 * L * H (block stride of a block-major pool)
  int64_t span_bytes;       // bytes moved per block: 2 * layer_count * H
  int64_t span_off;         // offset of the first moved layer in a block: 2 * layer0 * H
  int64_t units;            // total_blocks * tiles_per_block
  int64_t total_blocks;     // blocks in the plan
  int32_t n_segs;
  int32_t num_layers;
  int32_t layer0;           // first layer moved
  int32_t lines_per_chunk;  // H / line bytes (uniform path only)
  int32_t lines_per_block;  // ceil(span_bytes / line bytes)
  int32_t tiles_per_block;  // ceil(lines_per_block / unroll)
  uint32_t h_magic;         // division by H (per-lane path)
  uint32_t h_shift;
  int32_t order;            // 1 plan order, 2 blocks scattered, 3 tiles scattered,
                            // 4 tile-major over scattered blocks
  int64_t perm_mul;         // multiplier of the scattering permutation
};

struct XferArgs : XferShape {
  PoolArg src;
  PoolArg dst;
  flowkv_segment inline_runs[kInlineRuns];  // the plan, when it rides in the arguments
};
// The compiler appends 256 bytes of implicit arguments to every kernel's
// argument segment; the whole segment stays within 4 KiB.
constexpr size_t kImplicitArgBytes = 256;
static_assert(sizeof(XferArgs) + kImplicitArgBytes <= 4096,
              "kernel arguments must stay within 4 KiB");

// A plan in the planner's form (each run starting where the previous one
// ends) travels as 12-byte records, a run's length being the next record's
// `first` minus its own (total_blocks for the last).  With fewer base
// pointers than FLOWKV_MAX_LAYERS per side the kernel arguments hold longer
// plans: one pointer per side between block-major pools, one per layer (at
// most FLOWKV_INLINE_LAYERS) when a pool is layer-major.
struct CompactRun {
  int32_t src_block, dst_block, first;
};

template <int kBases>
struct PoolArgN {
  char* base[kBases];
  int64_t num_blocks;
};

template <int kBases, int kRuns>
struct XferArgsCompact : XferShape {
  static constexpr int kMaxBases = kBases;
  static constexpr int kMaxRuns = kRuns;
  PoolArgN<kBases> src;
  PoolArgN<kBases> dst;
  CompactRun inline_runs[kRuns];
};
using XferArgsBM = XferArgsCompact<1, FLOWKV_INLINE_RUNS_BLOCK_MAJOR>;
using XferArgsLM = XferArgsCompact<FLOWKV_INLINE_LAYERS, FLOWKV_INLINE_RUNS_LAYER_MAJOR>;
static_assert(sizeof(XferArgsBM) + kImplicitArgBytes <= 4096,
              "kernel arguments must stay within 4 KiB");
static_assert(sizeof(XferArgsLM) + kImplicitArgBytes <= 4096,
              "kernel arguments must stay within 4 KiB");

// Pool memory is global memory; naming the address space lets the compiler
// emit global (not flat) vector loads and stores with a scalar base.
typedef __attribute__((address_space(1))) u32x4 gvec;

__device__ __forceinline__ gvec* as_global(char* p) { return (gvec*)(p); }

typedef __attribute__((address_space(4))) const flowkv_segment cseg;

__device__ __forceinline__ flowkv_segment load_seg(const cseg* p) {
  flowkv_segment s;
  s.src_block = p->src_block;
  s.dst_block = p->dst_block;
  s.n_blocks = p->n_blocks;
  s.first = p->first;
  return s;
}

// kCache bit 0: nontemporal loads; bit 1: nontemporal stores.
template <int kCache>
__device__ __forceinline__ u32x4 load16(const gvec* p) {
  if constexpr (kCache & 1) return __builtin_nontemporal_load(p);
  else return *p;
}

template <int kCache>
__device__ __forceinline__ void store16(gvec* p, u32x4 v) {
  if constexpr (kCache & 2) __builtin_nontemporal_store(v, p);
  else *p = v;
}

// Start of line j (0 <= j < lines_per_block) of the moved span of block b
// when every line lies in one chunk: chunk r = j / lines_per_chunk (counted
// from layer0), line w = j % lines_per_chunk.
template <bool kLM, class P, class A>
__device__ __forceinline__ char* line_base(const P& p, const A& a, int64_t b,
                                           int32_t j, int32_t r, int32_t w, int64_t line) {
  if constexpr (kLM)
    return p.base[a.layer0 + (r >> 1)] + (int64_t(r & 1) * p.num_blocks + b) * a.chunk_bytes +
           int64_t(w) * line;
  else
    return p.base[0] + b * a.block_bytes + a.span_off + int64_t(j) * line;
}

// Tile t of a block when every line lies inside one chunk: all pointer
// arithmetic is uniform across the workgroup; each lane adds its 16 bytes.
template <bool kSrcLM, bool kDstLM, int kU, int kCache, class A>
__device__ __forceinline__ void copy_tile_uniform(const A& a, int64_t sb, int64_t db,
                                                  int32_t t, int tid, int64_t line) {
  const int32_t j0 = t * kU;
  int32_t r = j0 / a.lines_per_chunk;
  int32_t w = j0 - r * a.lines_per_chunk;
  if (j0 + kU <= a.lines_per_block) {
    // full tile: kU loads in flight, then kU stores, no branches between
    // chunk and in-chunk line of every line of the tile (branch-free), then
    // every layer base the tile needs, so those loads issue back to back
    int32_t rr[kU], ww[kU];
#pragma unroll
    for (int i = 0; i < kU; ++i) {
      rr[i] = r;
      ww[i] = w;
      const bool wrap = ++w == a.lines_per_chunk;
      r += wrap;
      w = wrap ? 0 : w;
    }
    char* sbase[kU];
    char* dbase[kU];
#pragma unroll
    for (int i = 0; i < kU; ++i) {
      sbase[i] = kSrcLM ? a.src.base[a.layer0 + (rr[i] >> 1)] : a.src.base[0] + a.span_off;
      dbase[i] = kDstLM ? a.dst.base[a.layer0 + (rr[i] >> 1)] : a.dst.base[0] + a.span_off;
    }
    const gvec* sp[kU];
    gvec* dp[kU];
#pragma unroll
    for (int i = 0; i < kU; ++i) {
      const int64_t j = j0 + i;
      sp[i] = as_global(kSrcLM ? sbase[i] + (int64_t(rr[i] & 1) * a.src.num_blocks + sb) * a.chunk_bytes + int64_t(ww[i]) * line
                               : sbase[i] + sb * a.block_bytes + j * line) + tid;
      dp[i] = as_global(kDstLM ? dbase[i] + (int64_t(rr[i] & 1) * a.dst.num_blocks + db) * a.chunk_bytes + int64_t(ww[i]) * line
                               : dbase[i] + db * a.block_bytes + j * line) + tid;
    }
    u32x4 v[kU];
#pragma unroll
    for (int i = 0; i < kU; ++i) v[i] = load16<kCache>(sp[i]);
#pragma unroll
    for (int i = 0; i < kU; ++i) store16<kCache>(dp[i], v[i]);
  } else {
    // the block's last, short tile
    for (int32_t j = j0; j < a.lines_per_block; ++j) {
      const u32x4 v = load16<kCache>(as_global(line_base<kSrcLM>(a.src, a, sb, j, r, w, line)) + tid);
      store16<kCache>(as_global(line_base<kDstLM>(a.dst, a, db, j, r, w, line)) + tid, v);
      if (++w == a.lines_per_chunk) {
        w = 0;
        ++r;
      }
    }
  }
}

__device__ __forceinline__ uint32_t div_by_h(uint32_t o, uint32_t magic, uint32_t shift) {
  const uint64_t hi = __umulhi(o, magic);
  return uint32_t((hi + o) >> shift);
}

// Byte o of the moved span of block b for any H (a multiple of 16): chunk
// r = o / H, counted from layer0.
template <bool kLM, class P, class A>
__device__ __forceinline__ char* byte_addr(const P& p, char* const* lds_base,
                                           const A& a, int64_t b, int64_t o) {
  if constexpr (kLM) {
    const uint32_t r = div_by_h(uint32_t(o), a.h_magic, a.h_shift);
    const int64_t w = o - int64_t(r) * a.chunk_bytes;
    return lds_base[a.layer0 + (r >> 1)] + (int64_t(r & 1) * p.num_blocks + b) * a.chunk_bytes + w;
  } else {
    return p.base[0] + b * a.block_bytes + a.span_off + o;
  }
}

// Tile t of a block for any H: each lane finds its own chunk.
template <bool kSrcLM, bool kDstLM, int kU, int kCache, class A>
__device__ __forceinline__ void copy_tile_lanes(const A& a, char* const* s_src,
                                                char* const* s_dst, int64_t sb, int64_t db,
                                                int32_t t, int tid, int64_t line) {
  const int64_t o0 = int64_t(t) * kU * line + int64_t(tid) * 16;
  if (int64_t(t + 1) * kU * line <= a.span_bytes) {
    const gvec* sp[kU];
    gvec* dp[kU];
#pragma unroll
    for (int i = 0; i < kU; ++i) {
      const int64_t o = o0 + int64_t(i) * line;
      sp[i] = as_global(byte_addr<kSrcLM>(a.src, s_src, a, sb, o));
      dp[i] = as_global(byte_addr<kDstLM>(a.dst, s_dst, a, db, o));
    }
    u32x4 v[kU];
#pragma unroll
    for (int i = 0; i < kU; ++i) v[i] = load16<kCache>(sp[i]);
#pragma unroll
    for (int i = 0; i < kU; ++i) store16<kCache>(dp[i], v[i]);
  } else {
    for (int64_t o = o0; o < a.span_bytes; o += line) {
      const u32x4 v = load16<kCache>(as_global(byte_addr<kSrcLM>(a.src, s_src, a, sb, o)));
      store16<kCache>(as_global(byte_addr<kDstLM>(a.dst, s_dst, a, db, o)), v);
    }
  }
}

// Record i of the plan: from device memory (read through the constant
// address space) or from the kernel arguments.  Both stay on the scalar unit.
template <bool kInline>
__device__ __forceinline__ int32_t run_first(const XferArgs& a, const cseg* segs, int32_t i) {
  if constexpr (kInline) return a.inline_runs[i].first;
  else return segs[i].first;
}

template <bool kInline>
__device__ __forceinline__ flowkv_segment run_at(const XferArgs& a, const cseg* segs, int32_t i) {
  if constexpr (kInline) return a.inline_runs[i];
  else return load_seg(segs + i);
}

// The compact inline forms: the same records, each run ending where the
// next one starts.
template <bool kInline, int B, int R>
__device__ __forceinline__ int32_t run_first(const XferArgsCompact<B, R>& a, const cseg*,
                                             int32_t i) {
  return a.inline_runs[i].first;
}

template <bool kInline, int B, int R>
__device__ __forceinline__ flowkv_segment run_at(const XferArgsCompact<B, R>& a, const cseg*,
                                                 int32_t i) {
  const CompactRun r = a.inline_runs[i];
  const int32_t end = i + 1 < a.n_segs ? a.inline_runs[i + 1].first : int32_t(a.total_blocks);
  return flowkv_segment{r.src_block, r.dst_block, end - r.first, r.first};
}

// Index of the last run whose first block is <= g, by galloping from run s
// (backward or forward) to a bracket [lo, hi) with first[lo] <= g < first[hi]
// and bisecting it.  Always returns an index in [0, n).
template <bool kInline, class A>
__device__ __forceinline__ int32_t find_run(const A& a, const cseg* segs, int32_t n,
                                            int64_t g, int32_t s) {
  int32_t lo, hi, step = 1;
  if (run_first<kInline>(a, segs, s) > g) {
    hi = s;
    lo = s - 1;
    while (lo > 0 && run_first<kInline>(a, segs, lo) > g) {
      hi = lo;
      step <<= 1;
      lo = hi - step > 0 ? hi - step : 0;
    }
    lo = lo > 0 ? lo : 0;
  } else {
    lo = s;
    hi = s + 1;
    while (hi < n && run_first<kInline>(a, segs, hi) <= g) {
      lo = hi;
      step <<= 1;
      hi = lo + step < n ? lo + step : n;
    }
  }
  while (hi - lo > 1) {
    const int32_t mid = (lo + hi) >> 1;
    if (run_first<kInline>(a, segs, mid) <= g) lo = mid;
    else hi = mid;
  }
  return lo;
}

// Where block g would sit if every run had the same length.
template <class A>
__device__ __forceinline__ int32_t guess_run(const A& a, int64_t g) {
  const int64_t s = g * a.n_segs / a.total_blocks;
  return int32_t(s < a.n_segs ? s : a.n_segs - 1);
}

template <bool kSrcLM, bool kDstLM, int kU, int kCache, bool kUniform, bool kInline,
          class A = XferArgs>
__global__ __launch_bounds__(1024) void kv_segment_copy(const A a) {
  __shared__ char* s_src[kUniform ? 1 : FLOWKV_MAX_LAYERS];
  __shared__ char* s_dst[kUniform ? 1 : FLOWKV_MAX_LAYERS];
  const int tid = threadIdx.x;
  const int64_t line = int64_t(blockDim.x) * 16;
  // Grid-stride over tiles (one tile per workgroup by default).  In plan
  // order the workgroups resident at one moment work on one window of
  // neighbouring tiles; the scattered orders spread them over the plan.
  int64_t u = blockIdx.x;
  if (u >= a.units) return;  // uniform across the workgroup
  if constexpr (!kUniform) {
    for (int l = tid; l < a.num_layers; l += blockDim.x) {
      s_src[l] = a.src.base[kSrcLM ? l : 0];
      s_dst[l] = a.dst.base[kDstLM ? l : 0];
    }
    __syncthreads();
  }

  // The plan is read-only for the whole launch: reading it through the
  // constant address space keeps the run lookups on the scalar unit.
  const cseg* segs = (const cseg*)(a.segs);
  const int64_t stride = gridDim.x;
  const int64_t g_step = stride / a.tiles_per_block;
  const int32_t t_step = int32_t(stride - g_step * a.tiles_per_block);
  // (gl, tl): block and tile of tile u in plan order, stepped incrementally
  int64_t gl = u / a.tiles_per_block;
  int32_t tl = int32_t(u - gl * a.tiles_per_block);
  int32_t s = -1;
  flowkv_segment seg{};
  for (; u < a.units; u += stride) {
    // the tile this iteration visits: plan order, or a fixed permutation of
    // blocks (2) or tiles (3) that scatters neighbouring workgroups, or tile
    // by tile over scattered blocks (4)
    int64_t g = gl;
    int32_t t = tl;
    if (a.order == 2) {
      g = gl * a.perm_mul % a.total_blocks;
    } else if (a.order == 3) {
      const int64_t v = u * a.perm_mul % a.units;
      g = v / a.tiles_per_block;
      t = int32_t(v - g * a.tiles_per_block);
    } else if (a.order == 4) {
      // tile-major: tile 0 of every block (blocks scattered), then tile 1 ...
      const int64_t tt = u / a.total_blocks;
      g = (u - tt * a.total_blocks) * a.perm_mul % a.total_blocks;
      t = int32_t(tt);
    }
    if (s < 0 || g < seg.first || g - seg.first >= int64_t(seg.n_blocks)) {
      s = find_run<kInline>(a, segs, a.n_segs, g, (s < 0 || a.order != 1) ? guess_run(a, g) : s);
      seg = run_at<kInline>(a, segs, s);
    }
    const int64_t off = g - seg.first;
    const int64_t sb = int64_t(seg.src_block) + off;
    const int64_t db = int64_t(seg.dst_block) + off;
    // a record that does not cover g, or points outside a pool, moves nothing
    const bool valid = off >= 0 && off < seg.n_blocks && sb >= 0 && sb < a.src.num_blocks &&
                       db >= 0 && db < a.dst.num_blocks;
    if (valid) {
      if constexpr (kUniform)
        copy_tile_uniform<kSrcLM, kDstLM, kU, kCache>(a, sb, db, t, tid, line);
      else
        copy_tile_lanes<kSrcLM, kDstLM, kU, kCache>(a, s_src, s_dst, sb, db, t, tid, line);
    }
    gl += g_step;
    tl += t_step;
    if (tl >= a.tiles_per_block) {
      tl -= a.tiles_per_block;
      ++gl;
    }
  }
}

template <class A>
using KernelOf = void (*)(A);
using KernelFn = KernelOf<XferArgs>;

template <class A, bool S, bool D, int U, int C, bool I>
KernelOf<A> pick_path(bool uniform) {
  return uniform ? kv_segment_copy<S, D, U, C, true, I, A>
                 : kv_segment_copy<S, D, U, C, false, I, A>;
}

template <class A, bool S, bool D, int U, bool I>
KernelOf<A> pick_cache(int cache, bool uniform) {
  switch (cache) {
    case 0: return pick_path<A, S, D, U, 0, I>(uniform);
    case 1: return pick_path<A, S, D, U, 1, I>(uniform);
    case 2: return pick_path<A, S, D, U, 2, I>(uniform);
    default: return pick_path<A, S, D, U, 3, I>(uniform);
  }
}

template <class A, bool S, bool D, bool I>
KernelOf<A> pick_unroll(int unroll, int cache, bool uniform) {
  switch (unroll) {
    case 2: return pick_cache<A, S, D, 2, I>(cache, uniform);
    case 4: return pick_cache<A, S, D, 4, I>(cache, uniform);
    case 8: return pick_cache<A, S, D, 8, I>(cache, uniform);
    default: return pick_cache<A, S, D, 16, I>(cache, uniform);
  }
}

template <bool I>
KernelFn pick_layouts(bool src_lm, bool dst_lm, int unroll, int cache, bool uniform) {
  if (src_lm && dst_lm) return pick_unroll<XferArgs, true, true, I>(unroll, cache, uniform);
  if (src_lm) return pick_unroll<XferArgs, true, false, I>(unroll, cache, uniform);
  if (dst_lm) return pick_unroll<XferArgs, false, true, I>(unroll, cache, uniform);
  return pick_unroll<XferArgs, false, false, I>(unroll, cache, uniform);
}

KernelFn pick_kernel(bool src_lm, bool dst_lm, int unroll, int cache, bool uniform, bool inl) {
  return inl ? pick_layouts<true>(src_lm, dst_lm, unroll, cache, uniform)
             : pick_layouts<false>(src_lm, dst_lm, unroll, cache, uniform);
}

// The compact inline forms: block-major pools on both sides, or a
// layer-major pool on at least one side.
KernelOf<XferArgsBM> pick_kernel_bm(int unroll, int cache, bool uniform) {
  return pick_unroll<XferArgsBM, false, false, true>(unroll, cache, uniform);
}

KernelOf<XferArgsLM> pick_kernel_lm(bool src_lm, bool dst_lm, int unroll, int cache,
                                    bool uniform) {
  if (src_lm && dst_lm) return pick_unroll<XferArgsLM, true, true, true>(unroll, cache, uniform);
  if (src_lm) return pick_unroll<XferArgsLM, true, false, true>(unroll, cache, uniform);
  return pick_unroll<XferArgsLM, false, true, true>(unroll, cache, uniform);
}

// Planner-form records the kernel arguments carry between two pools whose
// descriptors have been checked (0: only the general form).
int64_t compact_capacity(const flowkv_pool* src, const flowkv_pool* dst) {
  if (src->layout == FLOWKV_LAYOUT_BLOCK_MAJOR && dst->layout == FLOWKV_LAYOUT_BLOCK_MAJOR)
    return XferArgsBM::kMaxRuns;
  if (src->num_layers <= XferArgsLM::kMaxBases && dst->num_layers <= XferArgsLM::kMaxBases)
    return XferArgsLM::kMaxRuns;
  return 0;
}

// The compact arguments from the general ones and the planner's records.
template <class C>
C compact_args(const XferArgs& a, const flowkv_segment* runs, int64_t n) {
  C c{};
  static_cast<XferShape&>(c) = static_cast<const XferShape&>(a);
  const int nb = a.num_layers < C::kMaxBases ? a.num_layers : C::kMaxBases;
  for (int i = 0; i < nb; ++i) {
    c.src.base[i] = a.src.base[i];
    c.dst.base[i] = a.dst.base[i];
  }
  c.src.num_blocks = a.src.num_blocks;
  c.dst.num_blocks = a.dst.num_blocks;
  for (int64_t i = 0; i < n; ++i)
    c.inline_runs[i] = CompactRun{runs[i].src_block, runs[i].dst_block, runs[i].first};
  return c;
}

template <class A>
hipError_t launch_kernel(KernelOf<A> fn, A& args, int64_t grid, int threads, void* stream) {
  void* p[] = {&args};
  return hipLaunchKernel(reinterpret_cast<const void*>(fn), dim3(unsigned(grid)),
                         dim3(unsigned(threads)), p, 0, static_cast<hipStream_t>(stream));
}

// True when the records are the planner's form: run i starts where run i-1
// ends, every run holds a block, and the runs cover [0, total_blocks).
bool contiguous_plan(const flowkv_segment* r, int64_t n, int64_t total_blocks) {
  int64_t next = 0;
  for (int64_t i = 0; i < n; ++i) {
    if (r[i].first != next || r[i].n_blocks < 1) return false;
    next += r[i].n_blocks;
  }
  return next == total_blocks;
}

// Library defaults, from interleaved launch-shape comparisons over the five
// transfer workloads in both layouts: 1024 threads moving 4 vectors each per
// tile (64 KiB tiles), nontemporal loads and stores, one tile per workgroup.
// Visiting order: in plan order the resident workgroups of block-major pools
// stream one contiguous window of each pool, which ran 7-11% slower on the
// segment allocator's long runs.  Between two block-major pools the tiles are
// visited tile-major over scattered blocks (the resident workgroups then
// touch one 64 KiB piece each of many blocks): 0.3-1.2% faster than blocks
// scattered whole, except 0.4% slower on the 70B share.  With a layer-major
// pool on either side tile-major ran 13% slower, and blocks are scattered
// whole (a block's tiles then already span every layer tensor).
constexpr int kDefaultThreads = 1024;
constexpr int kDefaultUnroll = 4;
constexpr int kDefaultCache = 4;    // nontemporal loads and stores
constexpr int kDefaultOrder = 2;    // blocks scattered
constexpr int kDefaultOrderBM = 4;  // both pools block-major: tile-major
constexpr uint64_t kPermPrime = 2654435761ull;
constexpr int64_t kMaxGridPerCU = 2048;

std::atomic<int> g_cu_count[64];

int cu_count(int* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(FLOWKV_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev >= 0 && dev < 64) {
    int c = g_cu_count[dev].load(std::memory_order_relaxed);
    if (c > 0) {
      *out = c;
      return FLOWKV_OK;
    }
  }
  int c = 0;
  e = hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess || c <= 0)
    return fail(FLOWKV_EHIP, "CU count query: %s", hipGetErrorString(e));
  if (dev >= 0 && dev < 64) g_cu_count[dev].store(c, std::memory_order_relaxed);
  *out = c;
  return FLOWKV_OK;
}

struct Range {
  uintptr_t lo, hi;
};

int pool_ranges(const flowkv_pool* p, const char* name, Range* out, int* n) {
  if (!p) return fail(FLOWKV_EINVAL, "NULL %s pool", name);
  if (p->layout != FLOWKV_LAYOUT_LAYER_MAJOR && p->layout != FLOWKV_LAYOUT_BLOCK_MAJOR)
    return fail(FLOWKV_EINVAL, "%s pool: unknown layout %d", name, p->layout);
  if (p->num_layers < 1 || p->num_layers > FLOWKV_MAX_LAYERS)
    return fail(FLOWKV_EINVAL, "%s pool: %d layers, need 1..%d", name, p->num_layers,
                FLOWKV_MAX_LAYERS);
  if (p->num_blocks < 1) return fail(FLOWKV_EINVAL, "%s pool: %d blocks", name, p->num_blocks);
  if (p->reserved != 0) return fail(FLOWKV_EINVAL, "%s pool: reserved field not 0", name);
  if (p->chunk_bytes <= 0 || p->chunk_bytes % 16 != 0)
    return fail(FLOWKV_EINVAL, "%s pool: chunk_bytes %lld not a positive multiple of 16", name,
                (long long)p->chunk_bytes);
  const int64_t block_bytes = 2 * int64_t(p->num_layers) * p->chunk_bytes;
  if (block_bytes >= (int64_t(1) << 31))
    return fail(FLOWKV_EINVAL, "%s pool: block of %lld bytes, limit 2 GiB", name,
                (long long)block_bytes);
  if (!p->layer_base) return fail(FLOWKV_EINVAL, "%s pool: NULL layer_base", name);
  const bool lm = p->layout == FLOWKV_LAYOUT_LAYER_MAJOR;
  const int nb = lm ? p->num_layers : 1;
  const uint64_t bytes = lm ? uint64_t(2) * uint64_t(p->num_blocks) * uint64_t(p->chunk_bytes)
                            : uint64_t(p->num_blocks) * uint64_t(block_bytes);
  for (int i = 0; i < nb; ++i) {
    uintptr_t b = reinterpret_cast<uintptr_t>(p->layer_base[i]);
    if (!b) return fail(FLOWKV_EINVAL, "%s pool: NULL base pointer %d", name, i);
    if (b % 16) return fail(FLOWKV_EINVAL, "%s pool: base pointer %d not 16-byte aligned", name, i);
    out[i] = {b, b + uintptr_t(bytes)};
  }
  *n = nb;
  return FLOWKV_OK;
}

bool overlaps(const Range& x, const Range& y) { return x.lo < y.hi && y.lo < x.hi; }

}  // namespace

namespace {

int launch_transfer(const flowkv_pool* src, const flowkv_pool* dst,
                    const flowkv_segment* segs_dev, const flowkv_segment* segs_host,
                    int64_t n_segs, int64_t total_blocks, int32_t layer_begin,
                    int32_t layer_count, bool whole, const flowkv_launch_config* cfg,
                    void* hip_stream) {
  Range rs[FLOWKV_MAX_LAYERS], rd[FLOWKV_MAX_LAYERS];
  int ns = 0, nd = 0;
  int rc = pool_ranges(src, "sender", rs, &ns);
  if (!rc) rc = pool_ranges(dst, "receiver", rd, &nd);
  if (rc) return rc;
  if (src->num_layers != dst->num_layers || src->chunk_bytes != dst->chunk_bytes)
    return fail(FLOWKV_EINVAL, "pools disagree: %d vs %d layers, %lld vs %lld chunk bytes",
                src->num_layers, dst->num_layers, (long long)src->chunk_bytes,
                (long long)dst->chunk_bytes);
  for (int i = 0; i < ns; ++i)
    for (int j = 0; j < nd; ++j)
      if (overlaps(rs[i], rd[j]))
        return fail(FLOWKV_EINVAL, "sender tensor %d overlaps receiver tensor %d", i, j);
  for (int i = 0; i < nd; ++i)
    for (int j = i + 1; j < nd; ++j)
      if (overlaps(rd[i], rd[j]))
        return fail(FLOWKV_EINVAL, "receiver tensors %d and %d overlap", i, j);
  if (n_segs < 0 || total_blocks < 0)
    return fail(FLOWKV_EINVAL, "negative segment or block count");
  if (n_segs > INT32_MAX || total_blocks > INT32_MAX)
    return fail(FLOWKV_EINVAL, "segment or block count above 2^31-1");
  if (whole) {
    layer_begin = 0;
    layer_count = src->num_layers;
  }
  if (layer_begin < 0 || layer_count < 0 || layer_begin + int64_t(layer_count) > src->num_layers)
    return fail(FLOWKV_EINVAL, "layers [%d, %d + %d) outside the pools' %d layers", layer_begin,
                layer_begin, layer_count, src->num_layers);

  int threads = kDefaultThreads, unroll = kDefaultUnroll, cache = kDefaultCache, grid = 0;
  const bool both_bm =
      src->layout == FLOWKV_LAYOUT_BLOCK_MAJOR && dst->layout == FLOWKV_LAYOUT_BLOCK_MAJOR;
  int order = both_bm ? kDefaultOrderBM : kDefaultOrder;
  if (cfg) {
    if (cfg->threads) threads = cfg->threads;
    if (cfg->unroll) unroll = cfg->unroll;
    if (cfg->cache) cache = cfg->cache;
    if (cfg->order) order = cfg->order;
    grid = cfg->grid;
  }
  if (order < 1 || order > 4) return fail(FLOWKV_EINVAL, "order %d: need 1..4", order);
  if (threads < 64 || threads > 1024 || threads % 64)
    return fail(FLOWKV_EINVAL, "threads %d: need a multiple of 64 in 64..1024", threads);
  if (unroll != 2 && unroll != 4 && unroll != 8 && unroll != 16)
    return fail(FLOWKV_EINVAL, "unroll %d: need 2, 4, 8 or 16", unroll);
  if (cache < 1 || cache > 4) return fail(FLOWKV_EINVAL, "cache %d: need 1..4", cache);
  if (grid < 0) return fail(FLOWKV_EINVAL, "negative grid %d", grid);
  const bool inl = segs_host != nullptr;
  // more than kInlineRuns records ride in the kernel arguments only in a
  // compact form: the planner's records, between pools that need few base
  // pointers
  bool compact = false;
  if (inl && n_segs > kInlineRuns) {
    const int64_t cap = compact_capacity(src, dst);
    if (n_segs > cap)
      return fail(FLOWKV_ECAP,
                  "%lld runs: at most %lld travel in the kernel arguments between these pools "
                  "(%d for any plan; as the planner writes them, %d between block-major pools, "
                  "%d between pools of at most %d layers)",
                  (long long)n_segs, (long long)(cap > kInlineRuns ? cap : kInlineRuns),
                  kInlineRuns, XferArgsBM::kMaxRuns, XferArgsLM::kMaxRuns,
                  XferArgsLM::kMaxBases);
    if (!contiguous_plan(segs_host, n_segs, total_blocks))
      return fail(FLOWKV_ECAP,
                  "%lld runs: beyond %d, a plan travels in the kernel arguments only as the "
                  "planner writes it (each run starting where the previous one ends, the runs "
                  "covering total_blocks)",
                  (long long)n_segs, kInlineRuns);
    compact = true;
  }
  if (n_segs == 0 || total_blocks == 0 || layer_count == 0) return ok();
  if (!inl && !segs_dev) return fail(FLOWKV_EINVAL, "NULL segment list");
  if (!inl && reinterpret_cast<uintptr_t>(segs_dev) % 16)
    return fail(FLOWKV_EINVAL, "segment list not 16-byte aligned");

  XferArgs a{};
  for (int i = 0; i < ns; ++i) a.src.base[i] = static_cast<char*>(src->layer_base[i]);
  for (int i = 0; i < nd; ++i) a.dst.base[i] = static_cast<char*>(dst->layer_base[i]);
  a.src.num_blocks = src->num_blocks;
  a.dst.num_blocks = dst->num_blocks;
  a.segs = inl ? nullptr : segs_dev;
  if (inl)
    if (!compact)
      for (int64_t i = 0; i < n_segs; ++i) a.inline_runs[i] = segs_host[i];
  a.n_segs = int32_t(n_segs);
  a.num_layers = src->num_layers;
  a.chunk_bytes = src->chunk_bytes;
  a.block_bytes = 2 * int64_t(src->num_layers) * src->chunk_bytes;
  a.layer0 = layer_begin;
  a.span_off = 2 * int64_t(layer_begin) * src->chunk_bytes;
  a.span_bytes = 2 * int64_t(layer_count) * src->chunk_bytes;
  const int64_t line = int64_t(threads) * 16;
  const bool uniform = a.chunk_bytes % line == 0;
  a.lines_per_chunk = uniform ? int32_t(a.chunk_bytes / line) : 0;
  a.lines_per_block = int32_t((a.span_bytes + line - 1) / line);
  a.tiles_per_block = (a.lines_per_block + unroll - 1) / unroll;
  // division by H for the per-lane path: l = ceil(log2 H),
  // m = floor(2^32 (2^l - H) / H) + 1, q = (umulhi(o, m) + o) >> l
  {
    const uint64_t h = uint64_t(a.chunk_bytes);
    uint32_t l = 0;
    while ((uint64_t(1) << l) < h) ++l;
    a.h_shift = l;
    a.h_magic = uint32_t((((uint64_t(1) << l) - h) << 32) / h + 1);
  }
  a.units = total_blocks * int64_t(a.tiles_per_block);
  a.total_blocks = total_blocks;
  // scattering permutation x -> x * m mod M over blocks (M = total_blocks) or
  // tiles (M = units): m is a prime above 2^31 reduced mod M, so it is coprime
  // to every M < 2^31 and the map is a bijection; products stay below 2^62
  a.order = order;
  const int64_t perm_mod = order == 3 ? a.units : total_blocks;
  if (order != 1 && perm_mod >= (int64_t(1) << 31)) a.order = 1;
  a.perm_mul = int64_t(kPermPrime % uint64_t(perm_mod));

  // default: one tile per workgroup, at most kMaxGridPerCU workgroups per CU
  // (larger plans loop, grid stride)
  int64_t launch = a.units;
  if (grid == 0) {
    int cus = 0;
    rc = cu_count(&cus);
    if (rc) return rc;
    launch = std::min<int64_t>(launch, int64_t(cus) * kMaxGridPerCU);
  } else {
    launch = std::min<int64_t>(launch, grid);
  }
  launch = std::min<int64_t>(launch, INT32_MAX);

  const bool src_lm = src->layout == FLOWKV_LAYOUT_LAYER_MAJOR;
  const bool dst_lm = dst->layout == FLOWKV_LAYOUT_LAYER_MAJOR;
  hipError_t e;
  if (compact && both_bm) {
    XferArgsBM c = compact_args<XferArgsBM>(a, segs_host, n_segs);
    e = launch_kernel(pick_kernel_bm(unroll, cache - 1, uniform), c, launch, threads, hip_stream);
  } else if (compact) {
    XferArgsLM c = compact_args<XferArgsLM>(a, segs_host, n_segs);
    e = launch_kernel(pick_kernel_lm(src_lm, dst_lm, unroll, cache - 1, uniform), c, launch,
                      threads, hip_stream);
  } else {
    e = launch_kernel(pick_kernel(src_lm, dst_lm, unroll, cache - 1, uniform, inl), a, launch,
                      threads, hip_stream);
  }
  if (e == hipSuccess) e = hipGetLastError();
  if (e != hipSuccess) return fail(FLOWKV_EHIP, "kernel launch: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace

extern "C" int flowkv_transfer_ex(const flowkv_pool* src, const flowkv_pool* dst,
                                  const flowkv_segment* segs_dev, int64_t n_segs,
                                  int64_t total_blocks, const flowkv_launch_config* cfg,
                                  void* hip_stream) {
  return launch_transfer(src, dst, segs_dev, nullptr, n_segs, total_blocks, 0, 0, true, cfg,
                         hip_stream);
}

extern "C" int flowkv_transfer_inline(const flowkv_pool* src, const flowkv_pool* dst,
                                      const flowkv_segment* segs_host, int64_t n_segs,
                                      int64_t total_blocks, const flowkv_launch_config* cfg,
                                      void* hip_stream) {
  if (n_segs > 0 && !segs_host) return fail(FLOWKV_EINVAL, "NULL segment list");
  static const flowkv_segment none{};
  return launch_transfer(src, dst, nullptr, segs_host ? segs_host : &none, n_segs, total_blocks,
                         0, 0, true, cfg, hip_stream);
}

extern "C" int flowkv_inline_capacity(const flowkv_pool* src, const flowkv_pool* dst,
                                      int64_t* runs) {
  if (!src || !dst || !runs) return fail(FLOWKV_EINVAL, "NULL pool or output");
  const flowkv_pool* p[2] = {src, dst};
  for (const flowkv_pool* q : p) {
    if (q->layout != FLOWKV_LAYOUT_LAYER_MAJOR && q->layout != FLOWKV_LAYOUT_BLOCK_MAJOR)
      return fail(FLOWKV_EINVAL, "unknown layout %d", q->layout);
    if (q->num_layers < 1 || q->num_layers > FLOWKV_MAX_LAYERS)
      return fail(FLOWKV_EINVAL, "num_layers %d outside 1..%d", q->num_layers,
                  FLOWKV_MAX_LAYERS);
  }
  const int64_t cap = compact_capacity(src, dst);
  *runs = cap > kInlineRuns ? cap : kInlineRuns;
  return ok();
}

extern "C" int flowkv_transfer_layers(const flowkv_pool* src, const flowkv_pool* dst,
                                      const flowkv_segment* segs_dev, int64_t n_segs,
                                      int64_t total_blocks, int32_t layer_begin,
                                      int32_t layer_count, const flowkv_launch_config* cfg,
                                      void* hip_stream) {
  return launch_transfer(src, dst, segs_dev, nullptr, n_segs, total_blocks, layer_begin,
                         layer_count, false, cfg, hip_stream);
}

extern "C" int flowkv_transfer(const flowkv_pool* src, const flowkv_pool* dst,
                               const flowkv_segment* segs_dev, int64_t n_segs,
                               int64_t total_blocks, void* hip_stream) {
  return flowkv_transfer_ex(src, dst, segs_dev, n_segs, total_blocks, nullptr, hip_stream);
}
