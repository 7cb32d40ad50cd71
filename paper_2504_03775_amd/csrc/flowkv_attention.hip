// Paged decode attention over a FlowKV pool, for gfx950 (MI355X).
//
// FlowKV (arXiv 2504.03775), section 3.3, restructures the KV pool to the
// block-major (B, L, 2, H) layout of Eq. 5 so a transfer moves few large
// ranges, and adapts the PagedAttention kernel to read it.  This is that
// consumer: the decode step of Eq. 2 -- one new query token per request
// attending to the request's cached K and V of one layer -- reading either
// layout through the request's block list.  Grouped KV heads: Hq query heads
// share Hkv KV heads, query head h reading KV head h / (Hq / Hkv).
//
// Decode attention reads every cached K and V element once and does about
// G flops per byte (G = Hq / Hkv query heads per KV head): it is HBM-bound,
// and the work per token is kept small enough that the loads stay the limit.
// Two forms of pass 1 serve it: a vector-unit pass (below) for head_dim 64
// and for up to 4 query heads per KV head, and a matrix-core pass
// (decode_attn_split_mfma, further down) for 8 query heads per KV head at
// head_dim 128, where the vector pass reaches its ALU limit.
// Work split (flash-decoding style):
//   pass 1: one workgroup per (KV head, token split, request).  A token's
//           head vector (Dh bf16) is read by one 16-lane DPP row, Dh/16
//           values per lane; the workgroup's 32 rows take the split's tokens
//           round-robin, 4 tokens per row per step (with G = 8, two rows
//           share each token, 4 query heads each).  The loads are
//           branch-free, so their count per step is static.
//           - q.k: bf16 pair dot products (v_dot2) on the raw bf16 values.
//           - The 4 x (heads per row) partial scores of a row are summed
//             over its 16 lanes by a transposed butterfly (row mirror, half
//             mirror, two quad swaps): each step halves the values a lane
//             holds, so the row ends with every (token, head) score owned by
//             one lane (or replicated when there are fewer than 16).
//           - The owner lane runs the online softmax for its score: a
//             running reference max per head, moved only when a score
//             exceeds it by more than kLazy (log2 units), so unnormalised
//             weights stay <= 2^kLazy and the weighted sums are rarely
//             rescaled.
//           - The weights and rescale factors go through a small LDS row
//             buffer to all 16 lanes, which accumulate weight x V in float32.
//           Rows merge through LDS and the workgroup writes its partial
//           (reference max, sum, weighted V) per query head.
//   pass 2: one workgroup per (query head, request) merges the splits,
//           several splits per thread in flight.
// The grid covers every split up to the longest request.  When the caller
// passes the lengths on the host they ride in the kernel arguments (the
// kLens instantiations): a split past its request's end then leaves before
// any memory access and writes nothing, and pass 2 reads only the
// request's own splits.  Otherwise the lengths come from device memory and
// such a split leaves an empty record for pass 2.
// All arithmetic is float32; exponentials are exp2 of scores scaled by
// log2(e).  K and V are bfloat16; the output is float32.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <mutex>

#include "flowkv.h"
#include "flowkv_status.h"

using flowkv::fail;
using flowkv::ok;

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(1))) u32x4 gvec4;
typedef __attribute__((address_space(1))) u32x2 gvec2;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Pass-1 workgroups: 8 waves on the vector units, 4 on the matrix cores.
// (Eight waves per split, against four, took the 32-request batch from
// 0.246 to 0.239 ms at its 1024-token splits, measured interleaved.)
constexpr int kVecThreads = 512;
constexpr int kMfmaThreads = 256;
constexpr int kRowLanes = 16;              // lanes per token: one DPP row
constexpr int kRows = kVecThreads / kRowLanes;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLazy = 8.f;               // log2 of the largest unnormalised weight

// DPP lane patterns inside a 16-lane row
constexpr int kMirror = 0x140;             // lane i <- 15 - i
constexpr int kHalfMirror = 0x141;         // lane i <- 7 - i within each half
constexpr int kSwap1 = 0xB1;               // quad_perm [1,0,3,2]: i <- i ^ 1
constexpr int kSwap2 = 0x4E;               // quad_perm [2,3,0,1]: i <- i ^ 2
constexpr int kRor4 = 0x124;               // rotate the row by 4 lanes
constexpr int kRor8 = 0x128;               // rotate the row by 8 lanes

struct AttnArgs {
  const char* base[FLOWKV_MAX_LAYERS];  // pool tensors (layer-major) or base[0]
  int64_t pool_blocks;
  int64_t chunk_bytes;                  // bs * Hkv * Dh * 2
  int64_t block_bytes;                  // 2 * L * chunk_bytes
  const uint16_t* q;                    // (n_req, Hq, Dh) bf16
  const int32_t* tables;                // (n_req, max_blocks)
  const int32_t* seq_lens;              // (n_req)
  float* out;                           // (n_req, Hq, Dh) f32
  float* ws;                            // (n_req, Hq, max_splits, Dh + 2) f32
  int32_t layer, num_layers, block_size, kv_heads, q_heads, max_blocks;
  int32_t split_tokens, max_splits, max_seq_len;
  float scale_log2;                     // scale * log2(e)
  // the requests' lengths, when the caller passed them on the host (the
  // kernels instantiated with kLens read these instead of seq_lens)
  int32_t lens[FLOWKV_ATTN_INLINE_LENS];
};
// The compiler appends 256 bytes of implicit arguments; the whole segment
// stays within 4 KiB.
static_assert(sizeof(AttnArgs) + 256 <= 4096, "kernel arguments must stay within 4 KiB");

// Tokens of a request that take part: its length, capped by its block list
// and by max_seq_len (which also bounds the workspace's split count).
__device__ __forceinline__ int clamp_len(const AttnArgs& a, int T) {
  const int by_table = a.max_blocks * a.block_size;
  T = T < by_table ? T : by_table;
  return T < a.max_seq_len ? T : a.max_seq_len;
}

// Without the lengths in the arguments, a split at or past its request's end
// still leaves a record, an empty partial (max -inf, sum 0) for each of its
// kG query heads, so that the merge reads every split up to max_splits
// without the request's length.  Its weighted-V part is never written; the
// merge ignores it.
template <int kG, int kDh>
__device__ __forceinline__ void write_empty_partial(const AttnArgs& a, int g, int split, int r,
                                                    int tid) {
  if (tid < kG) {
    float* e = a.ws + ((int64_t(r) * a.q_heads + g * kG + tid) * a.max_splits + split) * (kDh + 2);
    e[0] = -INFINITY;
    e[1] = 0.f;
  }
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// by value: a bit cast of a vector-element lvalue would read element 0
__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t w) { return __builtin_bit_cast(bf16x2, w); }

template <int kCtrl>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), kCtrl, 0xF, 0xF, false));
}

// One butterfly step over partner pattern kCtrl.  With kN > 1 values the lane
// keeps half of them (the upper half when `upper`), adding the partner's
// copy of that half; the partner keeps the other half.  With one value it is
// a plain pairwise sum.
template <int kN, int kCtrl, int kP>
__device__ __forceinline__ void fold(float (&v)[kP], bool upper) {
  if constexpr (kN > 1) {
#pragma unroll
    for (int j = 0; j < kN / 2; ++j) {
      const float lo = v[j], hi = v[j + kN / 2];
      v[j] = (upper ? hi : lo) + dpp<kCtrl>(upper ? lo : hi);
    }
  } else {
    v[0] += dpp<kCtrl>(v[0]);
  }
}

template <int kW> struct Words;
template <> struct Words<4> {
  typedef u32x4 T;
  static __device__ __forceinline__ T load_nt(const char* p) {
    return __builtin_nontemporal_load((const gvec4*)p);
  }
};
template <> struct Words<2> {
  typedef u32x2 T;
  static __device__ __forceinline__ T load_nt(const char* p) {
    return __builtin_nontemporal_load((const gvec2*)p);
  }
};

template <int kDh, int kG, bool kLM, bool kLens>
__global__ __launch_bounds__(kVecThreads) void decode_attn_split(const AttnArgs a) {
  constexpr int kW = kDh / 32;                  // bf16 pairs per lane (4 or 2)
  constexpr int kV = 2 * kW;                    // K/V values per lane
  constexpr int kTok = 4;                       // tokens per row per step
  // With 8 query heads per KV head, two rows share each token, 4 heads each:
  // a lane then holds the state of 4 heads (the registers of 4 waves per
  // SIMD instead of 2); the pair's loads of the same token fall in one wave
  // instruction and cost no extra HBM traffic.
  constexpr int kHS = kG == 8 ? 2 : 1;          // rows per token
  constexpr int kGl = kG / kHS;                 // query heads per row
  constexpr int kTG = kRows / kHS;              // token groups per workgroup
  constexpr int kP = kTok * kGl;                // partial scores per lane per step
  constexpr int kR = kP > kRowLanes ? kP / kRowLanes : 1;  // scores a lane owns
  constexpr int kCS = (kGl + 3) / 4 * 4;        // rescale slots, padded to 16 B
  constexpr int kXS = kP + kCS;                 // LDS row buffer: weights, rescales
  constexpr int kStep = kTG * kTok;             // tokens per workgroup step
  using VT = typename Words<kW>::T;

  const int g = blockIdx.x;                     // KV head
  const int split = blockIdx.y;
  const int r = blockIdx.z;
  const int tid = threadIdx.x;
  const int row = tid / kRowLanes;
  const int lane = tid % kRowLanes;             // which kV values of the head vector
  const int tg = row / kHS;                     // the row's token group
  const int hh = row % kHS;                     // and its share of the heads

  const int t0 = split * a.split_tokens;
  const int bs = a.block_size;
  // with the length in the arguments, a split past the request's end leaves
  // at once, before any memory access, and writes no record
  if constexpr (kLens)
    if (t0 >= clamp_len(a, a.lens[r])) return;
  // the block IDs the split can touch, staged once in LDS: fetched without
  // waiting for the request's length (a split of at most
  // FLOWKV_ATTN_MAX_SPLIT tokens touches at most that many blocks plus one)
  __shared__ int32_t s_blk[FLOWKV_ATTN_MAX_SPLIT + 1];
  const int b0 = t0 / bs;
  {
    const int span = (t0 + a.split_tokens - 1) / bs - b0 + 1;
    const int nb = span < a.max_blocks - b0 ? span : a.max_blocks - b0;
    for (int i = tid; i < nb; i += kVecThreads)
      s_blk[i] = a.tables[int64_t(r) * a.max_blocks + b0 + i];
  }
  const int T = clamp_len(a, kLens ? a.lens[r] : a.seq_lens[r]);
  if (t0 >= T) {  // uniform: this split is past the request's end (no kLens)
    write_empty_partial<kG, kDh>(a, g, split, r, tid);
    return;
  }
  const int t1 = t0 + a.split_tokens < T ? t0 + a.split_tokens : T;

  // this lane's query pairs for each of the row's heads (raw bf16)
  const int h0 = g * kG + hh * kGl;             // the row's first query head
  uint32_t q[kGl][kW];
#pragma unroll
  for (int h = 0; h < kGl; ++h) {
    const uint32_t* qp = reinterpret_cast<const uint32_t*>(
        a.q + (int64_t(r) * a.q_heads + h0 + h) * kDh + lane * kV);
#pragma unroll
    for (int w = 0; w < kW; ++w) q[h][w] = qp[w];
  }

  // which partial score this lane owns after the butterfly: indices
  // own .. own + kR - 1 of the (token u, head h) list, index u * kGl + h
  int own = 0;
  {
    int n = kP;
    const int bits[4] = {8, 4, 1, 2};
#pragma unroll
    for (int s = 0; s < 4; ++s)
      if (n > 1) {
        if (lane & bits[s]) own += n / 2;
        n /= 2;
      }
  }
  const int u_own = own / kGl;                  // the owned scores' token

  // pool addressing: K of (block b, slot) at kbase + b * bstride + slot *
  // sstride + this lane's offset; V sits voff further
  const char* kbase;
  uint32_t bstride;
  int64_t voff;
  if constexpr (kLM) {
    kbase = a.base[a.layer];
    bstride = uint32_t(a.chunk_bytes);
    voff = a.pool_blocks * a.chunk_bytes;
  } else {
    kbase = a.base[0] + int64_t(a.layer) * 2 * a.chunk_bytes;
    bstride = uint32_t(a.block_bytes);
    voff = a.chunk_bytes;
  }
  const uint32_t sstride = uint32_t(a.kv_heads) * kDh * 2;
  kbase += g * kDh * 2 + lane * kV * 2;

  // token bookkeeping per step slot u: token index, its block (relative to
  // b0) and slot, advanced by kStep tokens per step without dividing
  int tok[kTok], bi[kTok], sl[kTok];
#pragma unroll
  for (int u = 0; u < kTok; ++u) {
    tok[u] = t0 + tg + u * kTG;
    bi[u] = tok[u] / bs - b0;
    sl[u] = tok[u] % bs;
  }
  const int step_q = kStep / bs, step_r = kStep % bs;

  __shared__ __attribute__((aligned(16))) float s_x[kRows][kXS];
  float acc[kGl][kV];
#pragma unroll
  for (int h = 0; h < kGl; ++h)
#pragma unroll
    for (int v = 0; v < kV; ++v) acc[h][v] = 0.f;
  float mref[kR], lsum[kR];
#pragma unroll
  for (int j = 0; j < kR; ++j) {
    mref[j] = -INFINITY;
    lsum[j] = 0.f;
  }
  __syncthreads();

  for (int base = t0; base < t1; base += kStep) {
    // K and V of each of the row's tokens that is in range and in the pool
    // (others stay zero, with their live bit clear); then the bookkeeping
    // advances one step.  (Issuing the next step's loads a step early
    // measured slower: its registers cost waves.)
    VT kw[kTok], vw[kTok];
    uint32_t live = 0;
#pragma unroll
    for (int u = 0; u < kTok; ++u) {
      // branch-free, so the loads' count is static: a token past the split's
      // end or with a block outside the pool reads the pool's first slot
      // instead, and its V is zeroed (its score is replaced by -inf below)
      const bool in = tok[u] < t1;
      const int b = s_blk[in ? bi[u] : 0];
      const bool ok = in && b >= 0 && b < a.pool_blocks;
      const char* kp =
          kbase + (ok ? uint64_t(uint32_t(b)) * bstride + uint32_t(sl[u]) * sstride : uint64_t(0));
      kw[u] = Words<kW>::load_nt(kp);
      vw[u] = Words<kW>::load_nt(kp + voff);
      if (!ok) vw[u] = VT{};
      live |= uint32_t(ok) << u;
      tok[u] += kStep;
      bi[u] += step_q;
      sl[u] += step_r;
      if (sl[u] >= bs) {
        sl[u] -= bs;
        bi[u] += 1;
      }
    }

    // partial q.k over this lane's values, index u * kGl + h
    float part[kP];
#pragma unroll
    for (int u = 0; u < kTok; ++u)
#pragma unroll
      for (int h = 0; h < kGl; ++h) {
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < kW; ++w)
          s = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(kw[u][w]), as_bf16x2(q[h][w]), s, false);
        part[u * kGl + h] = s;
      }
    fold<kP, kMirror>(part, lane & 8);
    fold<(kP / 2 > 1 ? kP / 2 : 1), kHalfMirror>(part, lane & 4);
    fold<(kP / 4 > 1 ? kP / 4 : 1), kSwap1>(part, lane & 1);
    fold<(kP / 8 > 1 ? kP / 8 : 1), kSwap2>(part, lane & 2);

    // owner lanes: online softmax per owned (token, head)
    const bool live_own = (live >> u_own) & 1u;
#pragma unroll
    for (int j = 0; j < kR; ++j) {
      const float sc = live_own ? part[j] * a.scale_log2 : -INFINITY;
      // the step's max over the 4 tokens of this head: the lanes holding
      // them differ only in lane bits 2 and 3
      float cm = fmaxf(sc, dpp<kRor4>(sc));
      cm = fmaxf(cm, dpp<kRor8>(cm));
      float c = 1.f;
      if (cm > mref[j] + kLazy) {  // also taken at the first live token (mref = -inf)
        c = __builtin_amdgcn_exp2f(mref[j] - cm);
        mref[j] = cm;
      }
      const float mu = mref[j] == -INFINITY ? 0.f : mref[j];
      const float p = __builtin_amdgcn_exp2f(sc - mu);
      lsum[j] = fmaf(lsum[j], c, p);
      s_x[row][own + j] = p;
      if (u_own == 0) s_x[row][kP + (own + j) % kGl] = c;
    }
    __builtin_amdgcn_wave_barrier();

    // every lane: rescale, then accumulate weight x V
    float px[kXS];
#pragma unroll
    for (int i = 0; i < kXS; i += 4) {
      const float4 x4 = *reinterpret_cast<const float4*>(&s_x[row][i]);
      px[i] = x4.x;
      px[i + 1] = x4.y;
      px[i + 2] = x4.z;
      px[i + 3] = x4.w;
    }
    bool rescale = false;
#pragma unroll
    for (int h = 0; h < kGl; ++h) rescale |= px[kP + h] != 1.f;
    if (rescale) {
#pragma unroll
      for (int h = 0; h < kGl; ++h)
#pragma unroll
        for (int v = 0; v < kV; ++v) acc[h][v] *= px[kP + h];
    }
#pragma unroll
    for (int u = 0; u < kTok; ++u) {
      float vf[kV];
#pragma unroll
      for (int w = 0; w < kW; ++w) {
        vf[2 * w] = bf16_lo(vw[u][w]);
        vf[2 * w + 1] = bf16_hi(vw[u][w]);
      }
#pragma unroll
      for (int h = 0; h < kGl; ++h)
#pragma unroll
        for (int v = 0; v < kV; ++v) acc[h][v] = fmaf(px[u * kGl + h], vf[v], acc[h][v]);
    }
    __builtin_amdgcn_wave_barrier();
  }

  // merge the rows that share heads: per head, a weight exp2(m_row - M) for
  // each row's reference max m_row against the largest M; a row that saw no
  // token has m_row = -inf and weighs nothing
  __shared__ float s_m[kRows][kGl], s_l[kRows][kGl], s_w[kRows][kGl];
  __shared__ __attribute__((aligned(16))) float s_acc[kVecThreads / 64][kG][kDh];
#pragma unroll
  for (int j = 0; j < kR; ++j) {
    float l = lsum[j];
    l += dpp<kRor4>(l);
    l += dpp<kRor8>(l);
    if (u_own == 0) {
      s_m[row][(own + j) % kGl] = mref[j];
      s_l[row][(own + j) % kGl] = l;
    }
  }
  __syncthreads();
  float* const dst0 = a.ws + ((int64_t(r) * a.q_heads + g * kG) * a.max_splits + split) * (kDh + 2);
  const int64_t head_stride = int64_t(a.max_splits) * (kDh + 2);
  if (tid < kG) {  // thread = query head of the group: rows x with x % kHS == its share
    const int sh = tid / kGl, h = tid % kGl;
    float M = -INFINITY;
    for (int x = sh; x < kRows; x += kHS) M = fmaxf(M, s_m[x][h]);
    float L = 0.f;
    for (int x = sh; x < kRows; x += kHS) {
      const float w = s_m[x][h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s_m[x][h] - M);
      s_w[x][h] = w;
      L = fmaf(s_l[x][h], w, L);
    }
    dst0[tid * head_stride] = M;
    dst0[tid * head_stride + 1] = L;
  }
  __syncthreads();
  // weight each row's sums, add the rows of a wave that share heads (lane
  // distance 16 x kHS), then the waves
  const int wave = tid / 64, row_in_wave = row % 4;
#pragma unroll
  for (int h = 0; h < kGl; ++h) {
    const float w = s_w[row][h];
#pragma unroll
    for (int v = 0; v < kV; ++v) {
      float x = acc[h][v] * w;
      if constexpr (kHS == 1) x += __shfl_xor(x, 16);
      x += __shfl_xor(x, 32);
      if (row_in_wave < kHS) s_acc[wave][hh * kGl + h][lane * kV + v] = x;
    }
  }
  __syncthreads();
  for (int i = tid; i < kG * kDh; i += kVecThreads) {
    const int h = i / kDh, d = i % kDh;
    float A = 0.f;
#pragma unroll
    for (int x = 0; x < kVecThreads / 64; ++x) A += s_acc[x][h][d];
    dst0[h * head_stride + 2 + d] = A;
  }
}

// Pass 1 on the matrix cores, head_dim 128 (FlowKV section 3.3's consumer,
// the same arithmetic as decode_attn_split up to rounding order).  Each wave
// takes its own tiles of 32 tokens; per tile:
//   - q.k: S (16 x 32, rows = query heads, padded past G) = Q (16 x 128) K^T
//     as 2 x 4 bf16 MFMAs (16x16x32).  A lane's K load is directly the B
//     operand: 16 bytes of one token (lane % 16) at dims 32 i + 8 (lane / 16).
//   - online softmax in the MFMA output layout: a lane holds 4 heads (rows
//     4 (lane / 16) + j) of 2 tokens; row maxima by DPP rotations over the
//     16-lane row; the same lazy reference max as the vector kernel.
//   - P goes through a small LDS transpose into the A operand and is split
//     into two bf16 parts (hi = bf16(P), lo = bf16(P - hi)), so P.V keeps
//     about 16 significant bits: O += P_hi V + P_lo V, 2 x 8 MFMAs.
//   - V lands in LDS straight from memory (global_load_lds, 16 bytes per
//     lane, no registers) and is read transposed as the B operand; the
//     contraction runs over tokens in the permuted order k = 8 q + e <->
//     token 4 e + q on both operands.  The compiler does not track these
//     loads for LDS reads, so the wave waits for them explicitly.
//   - the next tile's K and V loads are issued right after this tile's q.k,
//     into the wave's other V buffer, so they are in flight during this
//     tile's softmax and P.V (4% faster on a 70B share, measured).  With
//     the second buffer (78.6 KB of LDS in all), two workgroups fit on a
//     CU, not three: LDS, not the 168 registers per lane (136 vector, 32
//     accumulation), sets that limit.  None of the measured workloads ran
//     slower for it.
// The waves' partial (max, sum, weighted V) merge through LDS at the end.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int kCtrl>
__device__ __forceinline__ float dpp_max(float x) { return fmaxf(x, dpp<kCtrl>(x)); }

template <int kG, bool kLM, bool kLens>
__global__ __launch_bounds__(kMfmaThreads) void decode_attn_split_mfma(const AttnArgs a) {
  constexpr int kDh = 128;
  constexpr int kWaves = kMfmaThreads / 64;
  constexpr int kTile = 32;                      // tokens per wave step
  constexpr int kVBytes = 8 * 1024;              // LDS bytes of a wave's V tile
  constexpr int kStep = kWaves * kTile;          // tokens per workgroup step
  // What issue() puts in flight for one tile: each lane follows kLaneTokens
  // tokens (16 apart); a token's head vector (kDh bf16) is read by the 4 lanes
  // of one MFMA column group, 16 bytes each per instruction, so kTokLoads
  // instructions per token for K (into registers) and as many for V (into
  // LDS).  Every one of them counts once against the vector-memory counter.
  constexpr int kLaneTokens = kTile / 16;
  constexpr int kTokLoads = kDh * 2 / (4 * 16);
  constexpr int kIssueVm = kLaneTokens * kTokLoads * 2;
  static_assert(kLaneTokens == 2 && kTokLoads == 4, "issue() is written for 2 x 4 loads");
  static_assert(kIssueVm < 64, "the wait count must fit the 6-bit vector-memory counter");
  static_assert(kG == 4 || kG == 8, "matrix-core pass for 4 or 8 heads per KV head");
  const int g = blockIdx.x, split = blockIdx.y, r = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, ln = tid & 63;
  const int q4 = ln >> 4, c16 = ln & 15;         // MFMA lane coordinates

  const int t0 = split * a.split_tokens;
  const int bs = a.block_size;
  if constexpr (kLens)
    if (t0 >= clamp_len(a, a.lens[r])) return;
  __shared__ int32_t s_blk[FLOWKV_ATTN_MAX_SPLIT + 1];
  const int b0 = t0 / bs;
  {
    const int span = (t0 + a.split_tokens - 1) / bs - b0 + 1;
    const int nb = span < a.max_blocks - b0 ? span : a.max_blocks - b0;
    for (int i = tid; i < nb; i += kMfmaThreads)
      s_blk[i] = a.tables[int64_t(r) * a.max_blocks + b0 + i];
  }
  const int T = clamp_len(a, kLens ? a.lens[r] : a.seq_lens[r]);
  if (t0 >= T) {  // uniform: this split is past the request's end (no kLens)
    write_empty_partial<kG, kDh>(a, g, split, r, tid);
    return;
  }
  const int t1 = t0 + a.split_tokens < T ? t0 + a.split_tokens : T;

  // Q as the A operand of q.k: Q[head c16][32 i + 8 q4 .. + 8]; rows past G are zero
  bf16x8 qa[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    u32x4 w = u32x4{0, 0, 0, 0};
    if (c16 < kG)
      w = *reinterpret_cast<const u32x4*>(a.q + (int64_t(r) * a.q_heads + g * kG + c16) * kDh +
                                          32 * i + 8 * q4);
    qa[i] = __builtin_bit_cast(bf16x8, w);
  }

  const char* kbase;
  uint32_t bstride;
  int64_t voff;
  if constexpr (kLM) {
    kbase = a.base[a.layer];
    bstride = uint32_t(a.chunk_bytes);
    voff = a.pool_blocks * a.chunk_bytes;
  } else {
    kbase = a.base[0] + int64_t(a.layer) * 2 * a.chunk_bytes;
    bstride = uint32_t(a.block_bytes);
    voff = a.chunk_bytes;
  }
  const uint32_t sstride = uint32_t(a.kv_heads) * kDh * 2;
  kbase += g * kDh * 2 + 16 * q4;

  // each lane follows two tokens of its wave's tile: 16 gg + c16
  int tok[kLaneTokens], bi[kLaneTokens], sl[kLaneTokens];
#pragma unroll
  for (int gg = 0; gg < kLaneTokens; ++gg) {
    tok[gg] = t0 + wave * kTile + 16 * gg + c16;
    bi[gg] = tok[gg] / bs - b0;
    sl[gg] = tok[gg] % bs;
  }
  const int step_q = kStep / bs, step_r = kStep % bs;

  // LDS: per wave two V tiles, double-buffered (a tile is 8 blocks of 1 KB,
  // one per load instruction: block (gg, i) holds, at lane * 16, the 16 bytes
  // that lane loaded) and the P transpose; after the loop the V area holds
  // the waves' weighted sums
  __shared__ __attribute__((aligned(16))) uint8_t s_v[2 * kWaves * kVBytes];
  __shared__ __attribute__((aligned(16))) float s_pt[kWaves][16][kTile];
  static_assert(sizeof(float) * kWaves * kG * kDh <= sizeof(s_v), "merge area fits");
  uint8_t* const my_v0 = s_v + wave * kVBytes;
  uint8_t* const my_v1 = s_v + (kWaves + wave) * kVBytes;
  float(*const my_p)[kTile] = s_pt[wave];

  f32x4 o[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mref[4], lsum[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    mref[j] = -INFINITY;
    lsum[j] = 0.f;
  }
  __syncthreads();

  u32x4 kp[kLaneTokens][kTokLoads];
  bool live[kLaneTokens];
  // K of the lane's two tokens into registers, V into LDS buffer vbuf
  // (branch-free: a token past the end or outside the pool reads the pool's
  // first slot and is masked), then the bookkeeping advances one step.
  // Exactly kIssueVm vector-memory instructions, no other.
  auto issue = [&](uint8_t* vbuf) {
#pragma unroll
    for (int gg = 0; gg < kLaneTokens; ++gg) {
      const bool in = tok[gg] < t1;
      const int b = s_blk[in ? bi[gg] : 0];
      live[gg] = in && b >= 0 && b < a.pool_blocks;
      const char* kp0 = kbase + (live[gg] ? uint64_t(uint32_t(b)) * bstride +
                                                uint32_t(sl[gg]) * sstride
                                          : uint64_t(0));
      // cached, not nontemporal: each load reads half of a 128-byte line
      // and the next one the other half; with nontemporal loads the line
      // was often gone in between (9% more HBM traffic, measured)
#pragma unroll
      for (int i = 0; i < kTokLoads; ++i) {
        kp[gg][i] = *(const gvec4*)(kp0 + 64 * i);
        __builtin_amdgcn_global_load_lds(
            (const __attribute__((address_space(1))) void*)(kp0 + voff + 64 * i),
            (__attribute__((address_space(3))) void*)(vbuf + (gg * kTokLoads + i) * 1024), 16, 0,
            0);
      }
      tok[gg] += kStep;
      bi[gg] += step_q;
      sl[gg] += step_r;
      if (sl[gg] >= bs) {
        sl[gg] -= bs;
        bi[gg] += 1;
      }
    }
  };
  issue(my_v0);
  int cur = 0;
  for (int base = t0 + wave * kTile; base < t1; base += kStep) {
    uint8_t* const my_v = cur ? my_v1 : my_v0;
    // q.k: s[gg][j] = S[head 4 q4 + j][token 16 gg + c16]
    f32x4 s[2];
#pragma unroll
    for (int gg = 0; gg < 2; ++gg) {
      s[gg] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < 4; ++i)
        s[gg] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[i], __builtin_bit_cast(bf16x8, kp[gg][i]),
                                                        s[gg], 0, 0, 0);
    }
    // this tile's live flags, then the next tile's loads (into the other V
    // buffer), which overlap this tile's softmax and P.V
    const bool live_t[2] = {live[0], live[1]};
    issue(cur ? my_v0 : my_v1);
    // online softmax per head row
    bool rescale = false;
    float c[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float x0 = live_t[0] ? s[0][j] * a.scale_log2 : -INFINITY;
      const float x1 = live_t[1] ? s[1][j] * a.scale_log2 : -INFINITY;
      s[0][j] = x0;
      s[1][j] = x1;
      float cm = fmaxf(x0, x1);
      cm = dpp_max<kRor8>(cm);
      cm = dpp_max<kRor4>(cm);
      cm = dpp_max<0x122>(cm);   // rotate by 2
      cm = dpp_max<0x121>(cm);   // rotate by 1
      c[j] = 1.f;
      if (cm > mref[j] + kLazy) {
        c[j] = __builtin_amdgcn_exp2f(mref[j] - cm);
        mref[j] = cm;
        rescale = true;
      }
    }
    if (rescale) {
#pragma unroll
      for (int t = 0; t < 8; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) o[t][j] *= c[j];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float mu = mref[j] == -INFINITY ? 0.f : mref[j];
      const bool real = 4 * q4 + j < kG;
#pragma unroll
      for (int gg = 0; gg < 2; ++gg) {
        const float p = real ? __builtin_amdgcn_exp2f(s[gg][j] - mu) : 0.f;
        lsum[j] = fmaf(lsum[j], gg == 0 ? c[j] : 1.f, p);
        // P[head][token] at the A operand's position of token 16 gg + c16
        my_p[4 * q4 + j][8 * (c16 & 3) + 4 * gg + (c16 >> 2)] = p;
      }
    }
    __builtin_amdgcn_wave_barrier();

    // this tile's V is in LDS once every load but the next tile's kIssueVm
    // has returned; masked tokens' rows are then zeroed (their weight is 0,
    // and 0 x a stale NaN would not be)
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kIssueVm) : "memory");
    if (!live_t[0] || !live_t[1]) {
#pragma unroll
      for (int gg = 0; gg < 2; ++gg)
        if (!live_t[gg])
#pragma unroll
          for (int i = 0; i < kTokLoads; ++i)
            *reinterpret_cast<u32x4*>(my_v + (gg * kTokLoads + i) * 1024 + ln * 16) =
                u32x4{0, 0, 0, 0};
    }
    asm volatile("" ::: "memory");
    // A operand: P[head c16][k = 8 q4 + e], token 4 e + q4, split in two bf16
    bf16x8 ahi, alo;
    {
      const float4 p0 = *reinterpret_cast<const float4*>(&my_p[c16][8 * q4]);
      const float4 p1 = *reinterpret_cast<const float4*>(&my_p[c16][8 * q4 + 4]);
      const float pa[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const __bf16 h = (__bf16)pa[e];
        ahi[e] = h;
        alo[e] = (__bf16)(pa[e] - (float)h);
      }
    }
    // B operand per 16-dim tile: V[token 4 e + q4][dim 16 t + c16]
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      bf16x8 bv;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int tk = 4 * e + q4, bo = (16 * t + c16) * 2;
        bv[e] = *reinterpret_cast<const __bf16*>(
            my_v + ((tk >> 4) * 4 + (bo >> 6)) * 1024 + (16 * ((bo >> 4) & 3) + (tk & 15)) * 16 +
            (bo & 15));
      }
      o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ahi, bv, o[t], 0, 0, 0);
      o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(alo, bv, o[t], 0, 0, 0);
    }
    __builtin_amdgcn_wave_barrier();
    cur ^= 1;
  }
  // the loads issued for the tile after the last are still in flight
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // merge the 4 waves: per head a weight exp2(m_wave - M)
  __shared__ float s_m[kWaves][16], s_l[kWaves][16], s_w[kWaves][16];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float l = lsum[j];
    l += dpp<kRor8>(l);
    l += dpp<kRor4>(l);
    l += dpp<0x122>(l);
    l += dpp<0x121>(l);
    if (c16 == 0) {
      s_m[wave][4 * q4 + j] = mref[j];
      s_l[wave][4 * q4 + j] = l;
    }
  }
  __syncthreads();  // every wave is past the loop: the V area is free
  float* const s_o = reinterpret_cast<float*>(s_v);   // [wave][head < kG][dim]
#pragma unroll
  for (int t = 0; t < 8; ++t)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (4 * q4 + j < kG) s_o[(wave * kG + 4 * q4 + j) * kDh + 16 * t + c16] = o[t][j];
  float* const dst0 = a.ws + ((int64_t(r) * a.q_heads + g * kG) * a.max_splits + split) * (kDh + 2);
  const int64_t head_stride = int64_t(a.max_splits) * (kDh + 2);
  if (tid < kG) {
    float M = -INFINITY;
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][tid]);
    float L = 0.f;
    for (int w = 0; w < kWaves; ++w) {
      const float wt = s_m[w][tid] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s_m[w][tid] - M);
      s_w[w][tid] = wt;
      L = fmaf(s_l[w][tid], wt, L);
    }
    dst0[tid * head_stride] = M;
    dst0[tid * head_stride + 1] = L;
  }
  __syncthreads();
  for (int i = tid; i < kG * kDh; i += kMfmaThreads) {
    const int h = i / kDh, d = i % kDh;
    float A = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) A = fmaf(s_o[(w * kG + h) * kDh + d], s_w[w][h], A);
    dst0[h * head_stride + 2 + d] = A;
  }
}

// Pass 2: one workgroup per (query head, request).  Every split up to
// max_splits has a record (pass 1 leaves an empty one past a request's end;
// with kLens the merge reads only the request's own splits instead), so the
// merge needs no chain of dependent loads: a thread set of Dh threads takes
// every (256 / Dh)-th split, kMergeChunk splits' records loaded at once (all
// of them in one round for up to 256 / Dh x kMergeChunk splits), folded into
// a running (max, sum, weighted V) that is rescaled when its max rises; the
// sets then meet in LDS.
constexpr int kMergeThreads = 256;
constexpr int kMergeChunk = 16;

template <int kDh, bool kLens>
__global__ __launch_bounds__(kMergeThreads) void decode_attn_merge(const AttnArgs a) {
  constexpr int kParts = kMergeThreads / kDh;
  const int h = blockIdx.x, r = blockIdx.y, tid = threadIdx.x;
  const int d = tid % kDh, part = tid / kDh;
  // records per (request, head); with the lengths in the arguments only the
  // request's own splits hold one
  int ns = a.max_splits;
  if constexpr (kLens) ns = (clamp_len(a, a.lens[r]) + a.split_tokens - 1) / a.split_tokens;
  float* o = a.out + (int64_t(r) * a.q_heads + h) * kDh;
  const float* src = a.ws + (int64_t(r) * a.q_heads + h) * a.max_splits * (kDh + 2);
  float m = -INFINITY, l = 0.f, acc = 0.f;
  for (int x0 = part; x0 < ns; x0 += kParts * kMergeChunk) {
    // branch-free loads: a split past the end re-reads split 0 and is
    // masked; an empty record's weighted V (never written) is not used
    float ms[kMergeChunk], ls[kMergeChunk], vs[kMergeChunk];
#pragma unroll
    for (int j = 0; j < kMergeChunk; ++j) {
      const int x = x0 + j * kParts;
      const float* e = src + int64_t(x < ns ? x : 0) * (kDh + 2);
      ms[j] = e[0];
      ls[j] = e[1];
      vs[j] = e[2 + d];
      if (x >= ns) ms[j] = -INFINITY;
    }
    // no branch on the records' values, so every load above issues at once
    float cm = m;
#pragma unroll
    for (int j = 0; j < kMergeChunk; ++j) cm = fmaxf(cm, ms[j]);
    const float c = m == -INFINITY ? 0.f : exp2f(m - cm);  // 1 when the max holds
    l *= c;
    acc *= c;
#pragma unroll
    for (int j = 0; j < kMergeChunk; ++j) {
      const bool live = ms[j] != -INFINITY;
      const float w = live ? exp2f(ms[j] - cm) : 0.f;
      l = live ? fmaf(ls[j], w, l) : l;
      acc = live ? fmaf(vs[j], w, acc) : acc;
    }
    m = cm;
  }
  __shared__ float s_m[kParts], s_l[kParts];
  __shared__ float s_a[kParts][kDh];
  if (d == 0) {
    s_m[part] = m;
    s_l[part] = l;
  }
  s_a[part][d] = acc;
  __syncthreads();
  if (part == 0) {
    float M = -INFINITY;
#pragma unroll
    for (int p = 0; p < kParts; ++p) M = fmaxf(M, s_m[p]);
    float L = 0.f, A = 0.f;
#pragma unroll
    for (int p = 0; p < kParts; ++p) {
      if (s_m[p] != -INFINITY) {
        const float w = exp2f(s_m[p] - M);
        L = fmaf(s_l[p], w, L);
        A = fmaf(s_a[p][d], w, A);
      }
    }
    o[d] = L > 0.f ? A / L : 0.f;
  }
}

using SplitFn = void (*)(AttnArgs);

template <int D, bool LM, bool L>
SplitFn pick_group(int G) {
  switch (G) {
    case 1: return decode_attn_split<D, 1, LM, L>;
    case 2: return decode_attn_split<D, 2, LM, L>;
    case 4: return decode_attn_split<D, 4, LM, L>;
    default: return decode_attn_split<D, 8, LM, L>;
  }
}

// 8 query heads per KV head at head_dim 128: the matrix-core pass (the
// vector pass is near its ALU limit there)
bool matrix_core_pass(int D, int G) { return D == 128 && G == 8; }

template <bool L>
SplitFn pick_split_lens(int D, int G, bool lm) {
  if (matrix_core_pass(D, G))
    return lm ? decode_attn_split_mfma<8, true, L> : decode_attn_split_mfma<8, false, L>;
  if (D == 64) return lm ? pick_group<64, true, L>(G) : pick_group<64, false, L>(G);
  return lm ? pick_group<128, true, L>(G) : pick_group<128, false, L>(G);
}

SplitFn pick_split(int D, int G, bool lm, bool lens) {
  return lens ? pick_split_lens<true>(D, G, lm) : pick_split_lens<false>(D, G, lm);
}

const void* pick_merge(int D, bool lens) {
  if (D == 64)
    return lens ? reinterpret_cast<const void*>(decode_attn_merge<64, true>)
                : reinterpret_cast<const void*>(decode_attn_merge<64, false>);
  return lens ? reinterpret_cast<const void*>(decode_attn_merge<128, true>)
              : reinterpret_cast<const void*>(decode_attn_merge<128, false>);
}

int32_t auto_split(int32_t n_req, int32_t max_seq_len) {
  for (int32_t s = FLOWKV_ATTN_MIN_AUTO_SPLIT; s < FLOWKV_ATTN_MAX_SPLIT; s *= 2)
    if (int64_t(n_req) * ((int64_t(max_seq_len) + s - 1) / s) <= FLOWKV_ATTN_AUTO_PAIRS) return s;
  return FLOWKV_ATTN_MAX_SPLIT;
}

int64_t ws_bytes(int32_t n_req, int32_t q_heads, int32_t head_dim, int32_t max_seq_len,
                 int32_t split_tokens) {
  const int64_t splits = (int64_t(max_seq_len) + split_tokens - 1) / split_tokens;
  return int64_t(n_req) * q_heads * splits * (head_dim + 2) * int64_t(sizeof(float));
}

}  // namespace

extern "C" int flowkv_decode_attention_split(int32_t n_req, int32_t max_seq_len,
                                             int32_t* split_tokens) {
  if (!split_tokens) return fail(FLOWKV_EINVAL, "NULL output");
  if (n_req < 0 || max_seq_len < 0) return fail(FLOWKV_EINVAL, "negative sizes");
  *split_tokens = auto_split(n_req, max_seq_len);
  return ok();
}

extern "C" int flowkv_decode_attention_workspace(int32_t n_req, int32_t q_heads,
                                                 int32_t head_dim, int32_t max_seq_len,
                                                 int32_t split_tokens, int64_t* bytes) {
  if (!bytes) return fail(FLOWKV_EINVAL, "NULL output");
  if (n_req < 0 || q_heads < 1 || head_dim < 1 || max_seq_len < 0)
    return fail(FLOWKV_EINVAL, "bad attention shape");
  if (split_tokens == 0) split_tokens = auto_split(n_req, max_seq_len);
  if (split_tokens < 1 || split_tokens > FLOWKV_ATTN_MAX_SPLIT)
    return fail(FLOWKV_EINVAL, "split_tokens %d: need 1..%d", split_tokens,
                FLOWKV_ATTN_MAX_SPLIT);
  *bytes = ws_bytes(n_req, q_heads, head_dim, max_seq_len, split_tokens);
  return ok();
}

namespace {

// Checks every argument, then enqueues both passes with `ws` (ws_cap bytes)
// as the workspace.  When `scratch_ws` is set, the workspace is the library's
// own device array (found after the checks, so a call rejected on its
// arguments makes no runtime call) and a short capacity is reported as such.
int launch_attention(const flowkv_pool* pool, int32_t layer, const void* q_dev, int32_t n_req,
                     int32_t q_heads, int32_t kv_heads, int32_t head_dim,
                     const int32_t* block_tables_dev, int32_t max_blocks,
                     const int32_t* seq_lens_dev, const int32_t* seq_lens_host,
                     int32_t max_seq_len, float scale, int32_t split_tokens, float* out_dev,
                     void* ws, int64_t ws_cap, bool scratch_ws, void* hip_stream);

}  // namespace

extern "C" int flowkv_decode_attention(const flowkv_pool* pool, int32_t layer,
                                       const void* q_dev, int32_t n_req, int32_t q_heads,
                                       int32_t kv_heads, int32_t head_dim,
                                       const int32_t* block_tables_dev, int32_t max_blocks,
                                       const int32_t* seq_lens_dev,
                                       const int32_t* seq_lens_host, int32_t max_seq_len,
                                       float scale, int32_t split_tokens, float* out_dev,
                                       void* workspace_dev, int64_t workspace_bytes,
                                       void* hip_stream) {
  return launch_attention(pool, layer, q_dev, n_req, q_heads, kv_heads, head_dim,
                          block_tables_dev, max_blocks, seq_lens_dev, seq_lens_host,
                          max_seq_len, scale, split_tokens, out_dev, workspace_dev,
                          workspace_bytes, false, hip_stream);
}

// ---- the variant that allocates nothing --------------------------------------
//
// Its partial results live in `scratch`, a file-scope device array: each GPU
// the library runs on holds its own copy for the life of the process.  In
// host code `scratch` names a host-side stand-in, not device memory; the
// device address of the current GPU's copy comes from hipGetSymbolAddress,
// looked up once per device on its first call and kept in g_scratch_addr.
// Nothing in the array needs to start at zero: pass 1 writes every split
// record the merge reads.  Calls that overlap on one GPU share the array and
// race.
static __device__ __align__(256) float scratch[FLOWKV_ATTN_SCRATCH_BYTES / sizeof(float)];
static_assert(FLOWKV_ATTN_SCRATCH_BYTES % 256 == 0, "scratch size in whole 256-byte units");

namespace {

constexpr int kMaxDevices = 64;

std::atomic<void*> g_scratch_addr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of the current GPU's copy of `scratch`.
int scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(FLOWKV_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(FLOWKV_EINVAL, "device %d: the scratch table holds devices 0..%d", dev,
                kMaxDevices - 1);
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_addr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return fail(FLOWKV_EHIP, "scratch address on device %d: %s", dev,
                    hipGetErrorString(e));
      g_scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return FLOWKV_OK;
}

}  // namespace

extern "C" int flowkv_decode_attention_noalloc(const flowkv_pool* pool, int32_t layer,
                                               const void* q_dev, int32_t n_req,
                                               int32_t q_heads, int32_t kv_heads,
                                               int32_t head_dim,
                                               const int32_t* block_tables_dev,
                                               int32_t max_blocks, const int32_t* seq_lens_dev,
                                               const int32_t* seq_lens_host,
                                               int32_t max_seq_len, float scale,
                                               int32_t split_tokens, float* out_dev,
                                               void* hip_stream) {
  return launch_attention(pool, layer, q_dev, n_req, q_heads, kv_heads, head_dim,
                          block_tables_dev, max_blocks, seq_lens_dev, seq_lens_host,
                          max_seq_len, scale, split_tokens, out_dev, nullptr,
                          FLOWKV_ATTN_SCRATCH_BYTES, true, hip_stream);
}

namespace {

int launch_attention(const flowkv_pool* pool, int32_t layer, const void* q_dev, int32_t n_req,
                     int32_t q_heads, int32_t kv_heads, int32_t head_dim,
                     const int32_t* block_tables_dev, int32_t max_blocks,
                     const int32_t* seq_lens_dev, const int32_t* seq_lens_host,
                     int32_t max_seq_len, float scale, int32_t split_tokens, float* out_dev,
                     void* workspace_dev, int64_t workspace_bytes, bool scratch_ws,
                     void* hip_stream) {
  if (!pool) return fail(FLOWKV_EINVAL, "NULL pool");
  if (pool->layout != FLOWKV_LAYOUT_LAYER_MAJOR && pool->layout != FLOWKV_LAYOUT_BLOCK_MAJOR)
    return fail(FLOWKV_EINVAL, "unknown layout %d", pool->layout);
  if (pool->num_layers < 1 || pool->num_layers > FLOWKV_MAX_LAYERS || pool->num_blocks < 1 ||
      !pool->layer_base)
    return fail(FLOWKV_EINVAL, "bad pool descriptor");
  if (layer < 0 || layer >= pool->num_layers)
    return fail(FLOWKV_EINVAL, "layer %d outside the pool's %d layers", layer, pool->num_layers);
  if (head_dim != 64 && head_dim != 128)
    return fail(FLOWKV_EINVAL, "head_dim %d: need 64 or 128", head_dim);
  if (kv_heads < 1 || q_heads < 1 || q_heads % kv_heads)
    return fail(FLOWKV_EINVAL, "q_heads %d not a multiple of kv_heads %d", q_heads, kv_heads);
  const int G = q_heads / kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(FLOWKV_EINVAL, "query heads per KV head %d: need 1, 2, 4 or 8", G);
  const int64_t per_token = int64_t(kv_heads) * head_dim * 2;
  if (pool->chunk_bytes <= 0 || pool->chunk_bytes % per_token)
    return fail(FLOWKV_EINVAL, "chunk_bytes %lld is not block_size x %d KV heads x %d bf16",
                (long long)pool->chunk_bytes, kv_heads, head_dim);
  const int64_t bs = pool->chunk_bytes / per_token;
  // the kernel forms block offsets in 32 bits: one block stride under 4 GiB
  const int64_t stride = pool->layout == FLOWKV_LAYOUT_LAYER_MAJOR
                             ? pool->chunk_bytes
                             : 2 * int64_t(pool->num_layers) * pool->chunk_bytes;
  if (stride >= (int64_t(1) << 32))
    return fail(FLOWKV_EINVAL, "block stride of %lld bytes: need under 4 GiB", (long long)stride);
  if (n_req < 0 || max_blocks < 0 || max_seq_len < 0)
    return fail(FLOWKV_EINVAL, "negative sizes");
  // token indices are 32-bit in the kernels: a table row addresses at most
  // 2^31 - 1 tokens
  if (int64_t(max_blocks) * bs > INT32_MAX)
    return fail(FLOWKV_EINVAL, "max_blocks %d x block_size %lld tokens: need at most 2^31 - 1",
                max_blocks, (long long)bs);
  if (split_tokens == 0) split_tokens = auto_split(n_req, max_seq_len);
  if (split_tokens < 1 || split_tokens > FLOWKV_ATTN_MAX_SPLIT)
    return fail(FLOWKV_EINVAL, "split_tokens %d: need 1..%d", split_tokens,
                FLOWKV_ATTN_MAX_SPLIT);
  if (!(scale > 0.f) || !std::isfinite(scale)) return fail(FLOWKV_EINVAL, "bad scale");
  if (n_req == 0) return ok();
  const int64_t need = ws_bytes(n_req, q_heads, head_dim, max_seq_len, split_tokens);
  // (a workspace of 0 bytes, when max_seq_len is 0, may be NULL)
  // lengths from the host ride in the kernel arguments (then the device
  // copy is not read)
  const bool lens = seq_lens_host && n_req <= FLOWKV_ATTN_INLINE_LENS;
  if (!q_dev || !block_tables_dev || (!seq_lens_dev && !lens) || !out_dev ||
      (!scratch_ws && !workspace_dev && need > 0))
    return fail(FLOWKV_EINVAL, "NULL device pointer");
  if (workspace_bytes < need) {
    if (scratch_ws)
      return fail(FLOWKV_ECAP,
                  "%lld bytes of partial results needed, the library's scratch holds %lld "
                  "(fewer requests or query heads per call, or a longer split)",
                  (long long)need, (long long)workspace_bytes);
    return fail(FLOWKV_ECAP, "workspace of %lld bytes, %lld needed", (long long)workspace_bytes,
                (long long)need);
  }
  if (reinterpret_cast<uintptr_t>(q_dev) % 16)
    return fail(FLOWKV_EINVAL, "query not 16-byte aligned");
  // the launch grids put requests and splits on dimensions limited to 65,535
  const int64_t splits = (int64_t(max_seq_len) + split_tokens - 1) / split_tokens;
  if (n_req > 65535 || splits > 65535)
    return fail(FLOWKV_EINVAL, "%d requests, %lld splits: each must be at most 65535 per call",
                n_req, (long long)splits);
  const bool lm = pool->layout == FLOWKV_LAYOUT_LAYER_MAJOR;
  const int nbase = lm ? pool->num_layers : 1;
  AttnArgs a{};
  for (int i = 0; i < nbase; ++i) {
    if (!pool->layer_base[i] || reinterpret_cast<uintptr_t>(pool->layer_base[i]) % 16)
      return fail(FLOWKV_EINVAL, "pool base pointer %d NULL or not 16-byte aligned", i);
    a.base[i] = static_cast<const char*>(pool->layer_base[i]);
  }
  if (scratch_ws && need > 0) {
    const int rc = scratch_address(&workspace_dev);
    if (rc) return rc;
  }
  a.pool_blocks = pool->num_blocks;
  a.chunk_bytes = pool->chunk_bytes;
  a.block_bytes = 2 * int64_t(pool->num_layers) * pool->chunk_bytes;
  a.q = static_cast<const uint16_t*>(q_dev);
  a.tables = block_tables_dev;
  a.seq_lens = seq_lens_dev;
  a.out = out_dev;
  a.ws = static_cast<float*>(workspace_dev);
  a.layer = layer;
  a.num_layers = pool->num_layers;
  a.block_size = int32_t(bs);
  a.kv_heads = kv_heads;
  a.q_heads = q_heads;
  a.max_blocks = max_blocks;
  a.split_tokens = split_tokens;
  a.max_splits = int32_t((int64_t(max_seq_len) + split_tokens - 1) / split_tokens);
  a.max_seq_len = max_seq_len;
  a.scale_log2 = scale * kLog2e;
  if (lens)
    for (int32_t i = 0; i < n_req; ++i) a.lens[i] = seq_lens_host[i];
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  void* args[] = {&a};
  hipError_t e = hipSuccess;
  if (a.max_splits > 0) {
    SplitFn fn = pick_split(head_dim, G, lm, lens);
    e = hipLaunchKernel(reinterpret_cast<const void*>(fn),
                        dim3(unsigned(kv_heads), unsigned(a.max_splits), unsigned(n_req)),
                        dim3(matrix_core_pass(head_dim, G) ? kMfmaThreads : kVecThreads),
                        args, 0, st);
  }
  if (e == hipSuccess) {
    e = hipLaunchKernel(pick_merge(head_dim, lens), dim3(unsigned(q_heads), unsigned(n_req)),
                        dim3(kMergeThreads), args, 0, st);
  }
  if (e == hipSuccess) e = hipGetLastError();
  if (e != hipSuccess) return fail(FLOWKV_EHIP, "attention launch: %s", hipGetErrorString(e));
  return ok();
}

}  // namespace
