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
// Decode attention reads every cached K and V element once and does ~2
// flops per byte: it is HBM-bound, so it runs on the vector units (no MFMA).
// Work split (flash-decoding style):
//   pass 1: one workgroup per (KV head, token split, request).  A token's
//           head vector (Dh bf16 = 256 B at Dh 128) is read by a group of
//           Dh/8 lanes, 16 B each; the workgroup's groups take the split's
//           tokens round-robin, `kTok` tokens in flight per group, and keep
//           an online softmax (running max, sum, weighted V) per query head
//           of the KV group in registers.  Groups merge through LDS and the
//           workgroup writes its partial (max, sum, weighted V) per head.
//   pass 2: one workgroup per (query head, request) merges the splits.
// All arithmetic is float32; exponentials are exp2 of scores pre-scaled by
// log2(e).  K and V are bfloat16; the output is float32.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "flowkv.h"
#include "flowkv_status.h"

using flowkv::fail;
using flowkv::ok;

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) u32x4 gvec;

constexpr int kThreads = 256;       // pass-1 workgroup
constexpr int kTok = 4;             // tokens in flight per lane group
constexpr float kLog2e = 1.4426950408889634f;

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
};

// Tokens of a request that take part: its length, capped by its block list
// and by max_seq_len (which also bounds the workspace's split count).
__device__ __forceinline__ int clamp_len(const AttnArgs& a, int T) {
  const int by_table = a.max_blocks * a.block_size;
  T = T < by_table ? T : by_table;
  return T < a.max_seq_len ? T : a.max_seq_len;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Byte address of token slot `slot` of block b, K (kv 0) or V (kv 1), KV head
// g, in the pool's layout (Eq. 5): the slot holds Hkv x Dh values, head-major.
template <bool kLM, int kDh>
__device__ __forceinline__ const char* kv_addr(const AttnArgs& a, int64_t b, int kv, int slot,
                                               int g) {
  const int64_t in_chunk = (int64_t(slot) * a.kv_heads + g) * kDh * 2;
  if constexpr (kLM)
    return a.base[a.layer] + (int64_t(kv) * a.pool_blocks + b) * a.chunk_bytes + in_chunk;
  else
    return a.base[0] + b * a.block_bytes + (int64_t(a.layer) * 2 + kv) * a.chunk_bytes +
           in_chunk;
}

template <int kDh, int kG, bool kLM>
__global__ __launch_bounds__(kThreads) void decode_attn_split(const AttnArgs a) {
  constexpr int kLPT = kDh / 8;                 // lanes per token (8 values each)
  constexpr int kGroups = kThreads / kLPT;      // token groups per workgroup
  const int g = blockIdx.x;                     // KV head
  const int split = blockIdx.y;
  const int r = blockIdx.z;
  const int tid = threadIdx.x;
  const int grp = tid / kLPT;
  const int lane = tid % kLPT;                  // which 8 values of the head vector

  const int T = clamp_len(a, a.seq_lens[r]);
  const int t0 = split * a.split_tokens;
  if (t0 >= T) return;  // uniform: this split is past the request's end
  const int t1 = t0 + a.split_tokens < T ? t0 + a.split_tokens : T;

  // the split's block IDs, staged once in LDS (a split of at most
  // FLOWKV_ATTN_MAX_SPLIT tokens touches at most that many blocks plus one)
  __shared__ int32_t s_blk[FLOWKV_ATTN_MAX_SPLIT + 1];
  const int b0 = t0 / a.block_size;
  const int nb = (t1 - 1) / a.block_size - b0 + 1;
  for (int i = tid; i < nb; i += kThreads) s_blk[i] = a.tables[int64_t(r) * a.max_blocks + b0 + i];

  // this lane's 8 query values for each head of the KV group, pre-scaled
  float q[kG][8];
#pragma unroll
  for (int h = 0; h < kG; ++h) {
    const int qh = g * kG + h;
    const u32x4 w = *reinterpret_cast<const u32x4*>(a.q + (int64_t(r) * a.q_heads + qh) * kDh +
                                                    lane * 8);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      q[h][2 * j] = bf16_lo(w[j]) * a.scale_log2;
      q[h][2 * j + 1] = bf16_hi(w[j]) * a.scale_log2;
    }
  }
  __syncthreads();

  float m[kG], l[kG], acc[kG][8];
#pragma unroll
  for (int h = 0; h < kG; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[h][j] = 0.f;
  }

  for (int tb = t0 + grp; tb < t1; tb += kGroups * kTok) {
    u32x4 kw[kTok], vw[kTok];
    bool live[kTok];
#pragma unroll
    for (int u = 0; u < kTok; ++u) {
      const int t = tb + u * kGroups;
      kw[u] = u32x4{0, 0, 0, 0};
      vw[u] = u32x4{0, 0, 0, 0};
      live[u] = t < t1;
      if (live[u]) {
        const int64_t b = s_blk[t / a.block_size - b0];
        const bool in_pool = b >= 0 && b < a.pool_blocks;
        live[u] = in_pool;
        if (in_pool) {
          const int slot = t % a.block_size;
          kw[u] = __builtin_nontemporal_load((const gvec*)(kv_addr<kLM, kDh>(a, b, 0, slot, g)) +
                                             lane);
          vw[u] = __builtin_nontemporal_load((const gvec*)(kv_addr<kLM, kDh>(a, b, 1, slot, g)) +
                                             lane);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < kTok; ++u) {
      // the group's lanes all see the same `live`: t and b are per group
      float k[8], v[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        k[2 * j] = bf16_lo(kw[u][j]);
        k[2 * j + 1] = bf16_hi(kw[u][j]);
        v[2 * j] = bf16_lo(vw[u][j]);
        v[2 * j + 1] = bf16_hi(vw[u][j]);
      }
#pragma unroll
      for (int h = 0; h < kG; ++h) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) s = fmaf(q[h][j], k[j], s);
        // sum over the group's lanes (they are consecutive, kLPT a power of 2)
#pragma unroll
        for (int off = kLPT / 2; off > 0; off >>= 1) s += __shfl_xor(s, off, kLPT);
        if (live[u]) {
          const float m_new = fmaxf(m[h], s);
          const float c = exp2f(m[h] - m_new);
          const float p = exp2f(s - m_new);
          l[h] = l[h] * c + p;
#pragma unroll
          for (int j = 0; j < 8; ++j) acc[h][j] = fmaf(acc[h][j], c, p * v[j]);
          m[h] = m_new;
        }
      }
    }
  }

  // merge the token groups through LDS, one query head at a time; a group
  // that saw no token has m = -inf and weighs nothing
  __shared__ float s_m[kGroups];
  __shared__ float s_l[kGroups];
  __shared__ float s_acc[kGroups][kDh];
  const int ngrp_used = (t1 - t0) < kGroups ? (t1 - t0) : kGroups;
#pragma unroll
  for (int h = 0; h < kG; ++h) {
    if (lane == 0) {
      s_m[grp] = m[h];
      s_l[grp] = l[h];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) s_acc[grp][lane * 8 + j] = acc[h][j];
    __syncthreads();
    for (int d = tid; d < kDh; d += kThreads) {
      float M = -INFINITY;
      for (int x = 0; x < ngrp_used; ++x) M = fmaxf(M, s_m[x]);
      float L = 0.f, A = 0.f;
      for (int x = 0; x < ngrp_used; ++x) {
        const float w = s_m[x] == -INFINITY ? 0.f : exp2f(s_m[x] - M);
        L = fmaf(s_l[x], w, L);
        A = fmaf(s_acc[x][d], w, A);
      }
      float* dst =
          a.ws + ((int64_t(r) * a.q_heads + g * kG + h) * a.max_splits + split) * (kDh + 2);
      if (d == 0) {
        dst[0] = M;
        dst[1] = L;
      }
      dst[2 + d] = A;
    }
    __syncthreads();
  }
}

template <int kDh>
__global__ __launch_bounds__(kDh) void decode_attn_merge(const AttnArgs a) {
  const int h = blockIdx.x, r = blockIdx.y, d = threadIdx.x;
  const int T = clamp_len(a, a.seq_lens[r]);
  float* o = a.out + (int64_t(r) * a.q_heads + h) * kDh;
  if (T <= 0) {
    o[d] = 0.f;
    return;
  }
  const int ns = (T + a.split_tokens - 1) / a.split_tokens;
  const float* src = a.ws + (int64_t(r) * a.q_heads + h) * a.max_splits * (kDh + 2);
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, src[s * (kDh + 2)]);
  float L = 0.f, A = 0.f;
  for (int s = 0; s < ns; ++s) {
    const float ms = src[s * (kDh + 2)];
    const float w = ms == -INFINITY ? 0.f : exp2f(ms - M);
    L = fmaf(src[s * (kDh + 2) + 1], w, L);
    A = fmaf(src[s * (kDh + 2) + 2 + d], w, A);
  }
  o[d] = L > 0.f ? A / L : 0.f;
}

using SplitFn = void (*)(AttnArgs);

template <int D, bool LM>
SplitFn pick_group(int G) {
  switch (G) {
    case 1: return decode_attn_split<D, 1, LM>;
    case 2: return decode_attn_split<D, 2, LM>;
    case 4: return decode_attn_split<D, 4, LM>;
    default: return decode_attn_split<D, 8, LM>;
  }
}

SplitFn pick_split(int D, int G, bool lm) {
  if (D == 64) return lm ? pick_group<64, true>(G) : pick_group<64, false>(G);
  return lm ? pick_group<128, true>(G) : pick_group<128, false>(G);
}

int64_t ws_bytes(int32_t n_req, int32_t q_heads, int32_t head_dim, int32_t max_seq_len,
                 int32_t split_tokens) {
  const int64_t splits = (int64_t(max_seq_len) + split_tokens - 1) / split_tokens;
  return int64_t(n_req) * q_heads * splits * (head_dim + 2) * int64_t(sizeof(float));
}

}  // namespace

extern "C" int flowkv_decode_attention_workspace(int32_t n_req, int32_t q_heads,
                                                 int32_t head_dim, int32_t max_seq_len,
                                                 int32_t split_tokens, int64_t* bytes) {
  if (!bytes) return fail(FLOWKV_EINVAL, "NULL output");
  if (n_req < 0 || q_heads < 1 || head_dim < 1 || max_seq_len < 0)
    return fail(FLOWKV_EINVAL, "bad attention shape");
  if (split_tokens == 0) split_tokens = FLOWKV_ATTN_DEFAULT_SPLIT;
  if (split_tokens < 1 || split_tokens > FLOWKV_ATTN_MAX_SPLIT)
    return fail(FLOWKV_EINVAL, "split_tokens %d: need 1..%d", split_tokens,
                FLOWKV_ATTN_MAX_SPLIT);
  *bytes = ws_bytes(n_req, q_heads, head_dim, max_seq_len, split_tokens);
  return ok();
}

extern "C" int flowkv_decode_attention(const flowkv_pool* pool, int32_t layer,
                                       const void* q_dev, int32_t n_req, int32_t q_heads,
                                       int32_t kv_heads, int32_t head_dim,
                                       const int32_t* block_tables_dev, int32_t max_blocks,
                                       const int32_t* seq_lens_dev, int32_t max_seq_len,
                                       float scale, int32_t split_tokens, float* out_dev,
                                       void* workspace_dev, int64_t workspace_bytes,
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
  if (n_req < 0 || max_blocks < 0 || max_seq_len < 0)
    return fail(FLOWKV_EINVAL, "negative sizes");
  if (split_tokens == 0) split_tokens = FLOWKV_ATTN_DEFAULT_SPLIT;
  if (split_tokens < 1 || split_tokens > FLOWKV_ATTN_MAX_SPLIT)
    return fail(FLOWKV_EINVAL, "split_tokens %d: need 1..%d", split_tokens,
                FLOWKV_ATTN_MAX_SPLIT);
  if (!(scale > 0.f) || !std::isfinite(scale)) return fail(FLOWKV_EINVAL, "bad scale");
  if (n_req == 0) return ok();
  if (!q_dev || !block_tables_dev || !seq_lens_dev || !out_dev || !workspace_dev)
    return fail(FLOWKV_EINVAL, "NULL device pointer");
  const int64_t need = ws_bytes(n_req, q_heads, head_dim, max_seq_len, split_tokens);
  if (workspace_bytes < need)
    return fail(FLOWKV_ECAP, "workspace of %lld bytes, %lld needed", (long long)workspace_bytes,
                (long long)need);
  if (reinterpret_cast<uintptr_t>(q_dev) % 16)
    return fail(FLOWKV_EINVAL, "query not 16-byte aligned");
  const bool lm = pool->layout == FLOWKV_LAYOUT_LAYER_MAJOR;
  const int nbase = lm ? pool->num_layers : 1;
  AttnArgs a{};
  for (int i = 0; i < nbase; ++i) {
    if (!pool->layer_base[i] || reinterpret_cast<uintptr_t>(pool->layer_base[i]) % 16)
      return fail(FLOWKV_EINVAL, "pool base pointer %d NULL or not 16-byte aligned", i);
    a.base[i] = static_cast<const char*>(pool->layer_base[i]);
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
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  void* args[] = {&a};
  hipError_t e = hipSuccess;
  if (a.max_splits > 0) {
    SplitFn fn = pick_split(head_dim, G, lm);
    e = hipLaunchKernel(reinterpret_cast<const void*>(fn),
                        dim3(unsigned(kv_heads), unsigned(a.max_splits), unsigned(n_req)),
                        dim3(kThreads), args, 0, st);
  }
  if (e == hipSuccess) {
    const void* merge = head_dim == 64 ? reinterpret_cast<const void*>(decode_attn_merge<64>)
                                       : reinterpret_cast<const void*>(decode_attn_merge<128>);
    e = hipLaunchKernel(merge, dim3(unsigned(q_heads), unsigned(n_req)), dim3(unsigned(head_dim)),
                        args, 0, st);
  }
  if (e == hipSuccess) e = hipGetLastError();
  if (e != hipSuccess) return fail(FLOWKV_EHIP, "attention launch: %s", hipGetErrorString(e));
  return ok();
}
