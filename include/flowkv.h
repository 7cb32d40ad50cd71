/*
 * flowkv.h -- C ABI of the MI355X (gfx950) KV-cache transfer library.
 *
 * FlowKV (arXiv 2504.03775), section 3.3: after prefill, a request's KV cache
 * (K and V of every layer, in fixed-size paged blocks) moves from the prefill
 * side's block pool to the decode side's block pool.  Three pieces cut the
 * number of transfer operations that scattered blocks cause:
 *
 *   flowkv_alloc*  -- a segment-based allocator that places a request in as few
 *                     contiguous runs of block IDs as it can (section 3.3,
 *                     allocator paragraph);
 *   flowkv_plan*   -- bidirectional segment alignment: the runs of the request
 *                     whose block IDs step by one on the sending and the
 *                     receiving side together (section 3.3; Figure 3 caption);
 *   flowkv_transfer -- one device launch that copies every run of every layer's
 *                     K and V, in the per-layer layout (L, 2, B, H) or the
 *                     block-major layout (B, L, 2, H) of Eq. 5, on one GPU;
 *                     flowkv_transfer_request plans and launches one request
 *                     in a single call.
 *
 * Beside them: flowkv_decode_attention*, the paged decode attention that
 * reads either layout (the PagedAttention kernel section 3.3 adapts), and
 * flowkv_sched*, the load-aware scheduler of section 3.4 (Algorithm 1),
 * host only.
 *
 * Conventions for every entry point:
 *   - Functions return FLOWKV_OK (0) or a negative FLOWKV_E* code; nothing
 *     throws across the ABI.  flowkv_strerror() names a code;
 *     flowkv_last_error() gives the calling thread's last detailed message.
 *   - On error, output arguments are left untouched, except *n_out of the
 *     planners and *n_runs of flowkv_transfer_request on FLOWKV_ECAP.
 *   - The caller owns every buffer.  The library allocates no device memory and
 *     keeps no pointer after a call returns, except inside an allocator or a
 *     scheduler handle, and except the fixed scratch array of
 *     flowkv_decode_attention_noalloc (a static device array of the library's
 *     code object, not an allocation).
 *   - Block IDs and counts are int32; byte sizes and offsets are 64-bit.
 *   - Allocator and scheduler handles are not thread-safe; planners, the
 *     transfer and attention are reentrant.
 */
#ifndef FLOWKV_H
#define FLOWKV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------------- */
enum {
  FLOWKV_OK = 0,
  FLOWKV_EINVAL = -1, /* bad argument: NULL pointer, negative count, bad layout,
                         misaligned or overlapping pools, unknown policy      */
  FLOWKV_ENOSPC = -2, /* fewer free blocks than asked; allocator unchanged    */
  FLOWKV_ERANGE = -3, /* a block ID outside [0, pool blocks)                  */
  FLOWKV_EDUP = -4,   /* a block ID repeated where it must be unique, freeing
                         a free block, or marking a used block               */
  FLOWKV_ECAP = -5,   /* output capacity too small; *n_out holds the need     */
  FLOWKV_EHIP = -6,   /* the HIP runtime refused the launch                   */
  FLOWKV_ENOMEM = -7  /* host memory ran out; an allocator or scheduler handle
                         that returned it may be inconsistent: destroy it     */
};

/* ---- allocator policies ---------------------------------------------------- */
enum {
  /* Section 3.3 allocator: free blocks kept as maximal free runs; a request
     takes the best-fitting run (shortest run that holds it, lowest start on
     ties, blocks from its head); if no run holds it, it takes the longest runs
     whole (lowest start on ties) until the rest fits one run, which is then
     best-fitted -- the fewest runs any placement can use.  Freed blocks merge
     with free neighbours. */
  FLOWKV_POLICY_SEGMENT = 0,
  /* Naive free list the paper contrasts with: FIFO of free IDs, ascending at
     creation; alloc pops from the front, free appends in table order. */
  FLOWKV_POLICY_FIFO_SORTED = 1,
  /* Same FIFO, but starting as a seeded Fisher-Yates shuffle drawn from
     SplitMix64 (Steele, Lea, Flood 2014): for i = P-1 down to 1, swap slot i
     with slot next() mod (i+1), the generator state starting at the seed. */
  FLOWKV_POLICY_FIFO_SHUFFLED = 2
};

/* ---- pool layouts (Eq. 5) -------------------------------------------------- */
enum {
  /* (L, 2, B, H): one device tensor per layer, each (2, B, H) -- K blocks then
     V blocks.  layer_base[l] points at layer l's tensor. */
  FLOWKV_LAYOUT_LAYER_MAJOR = 0,
  /* (B, L, 2, H): one device tensor; a block's K and V of every layer are
     adjacent.  layer_base[0] points at it. */
  FLOWKV_LAYOUT_BLOCK_MAJOR = 1
};

#define FLOWKV_MAX_LAYERS 128
#define FLOWKV_INLINE_RUNS 64 /* plan records flowkv_transfer_inline carries */
#define FLOWKV_INLINE_RUNS_BLOCK_MAJOR 300 /* ... between two block-major pools, as
                                              the planner writes them */
#define FLOWKV_INLINE_LAYERS 32 /* pools of at most this many layers ...     */
#define FLOWKV_INLINE_RUNS_LAYER_MAJOR 264 /* ... carry this many planner-form
                                              records when either is layer-major */

typedef struct flowkv_allocator flowkv_allocator; /* opaque, host memory only */

/* One aligned run: n_blocks blocks starting at src_block on the sender and at
   dst_block on the receiver, all stepping by one together.  `first` is the
   run's position in the plan's block order: the sum of n_blocks over all
   earlier records of the same plan (a request's or a batch's), so a plan's
   records tile [0, total blocks) in order.  16 bytes, 16-byte aligned.

   The fourth field is `first`, not the index of the request a batch record
   belongs to: the kernel finds the run that holds a block by searching
   `first`, and the request index follows from it.  Runs never cross
   requests, so with flowkv_plan_batch's offsets the record belongs to the
   request r with offsets[r] <= first < offsets[r + 1] -- the last r with
   offsets[r] <= first, which skips requests with no blocks -- and covers its
   blocks first - offsets[r] .. + n_blocks - 1. */
typedef struct flowkv_segment {
  int32_t src_block;
  int32_t dst_block;
  int32_t n_blocks;
  int32_t first;
} flowkv_segment;

typedef struct flowkv_alloc_stats {
  int64_t free_blocks;   /* blocks not in use                         */
  int64_t free_segments; /* maximal runs of free block IDs            */
  int64_t largest_free;  /* blocks in the longest free run            */
} flowkv_alloc_stats;

/* A paged KV pool on the device.  chunk_bytes is H times the element size:
   the bytes of one (block, layer, K-or-V) slab, block_size tokens of
   kv_heads x head_dim elements each.  A block holds 2 * num_layers chunks. */
typedef struct flowkv_pool {
  int32_t layout;          /* FLOWKV_LAYOUT_*                                 */
  int32_t num_layers;      /* L, 1 .. FLOWKV_MAX_LAYERS                       */
  int32_t num_blocks;      /* B, >= 1                                         */
  int32_t reserved;        /* must be 0                                       */
  int64_t chunk_bytes;     /* > 0, a multiple of 16                           */
  void* const* layer_base; /* host array of device pointers, 16-byte aligned:
                              num_layers entries (layer-major) or 1 entry
                              (block-major)                                  */
} flowkv_pool;

/* Optional launch shape for flowkv_transfer_ex; a zero field takes the
   library's choice (order: 4 between two block-major pools, else 2).
   threads: workgroup size, a multiple of 64 in 64..1024.
   unroll:  16-byte vectors each thread moves per tile: 2, 4, 8 or 16.
   grid:    workgroups to launch, >= 1 (capped at the number of tiles).
   cache:   1 = plain loads and stores, 2 = nontemporal loads,
            3 = nontemporal stores, 4 = nontemporal loads and stores.
   order:   the order workgroups visit tiles in: 1 = plan order, 2 = blocks
            scattered by a fixed permutation (a block's tiles stay together),
            3 = tiles scattered by a fixed permutation, 4 = tile-major: tile 0
            of every block (blocks scattered as in 2), then tile 1, and so on.
            Same result for all. */
typedef struct flowkv_launch_config {
  int32_t threads;
  int32_t unroll;
  int32_t grid;
  int32_t cache;
  int32_t order;
} flowkv_launch_config;

/* ---- allocator (section 3.3, allocator paragraph) -------------------------- */

/* Create an allocator over block IDs [0, num_blocks), all free.  `seed` is used
   by FLOWKV_POLICY_FIFO_SHUFFLED only.  *out receives the handle.
   EINVAL: num_blocks < 0, unknown policy, out == NULL.  ENOMEM: host memory
   ran out (nothing is created).  The other allocator and planner calls also
   return ENOMEM if host memory runs out mid-call (see the status codes). */
int flowkv_allocator_create(int32_t num_blocks, int32_t policy, uint64_t seed,
                            flowkv_allocator** out);

/* Release the handle (NULL is accepted). */
void flowkv_allocator_destroy(flowkv_allocator* a);

/* Allocate n_blocks blocks; out_ids[0 .. n_blocks) receives them in the
   request's logical order.  All or nothing: ENOSPC when fewer are free, with
   the allocator unchanged.  n_blocks == 0 succeeds and writes nothing.
   EINVAL: a or out_ids NULL (out_ids may be NULL when n_blocks == 0),
   n_blocks < 0. */
int flowkv_alloc(flowkv_allocator* a, int32_t n_blocks, int32_t* out_ids);

/* Return ids[0 .. n) to the free pool, merging with free neighbours.
   ERANGE: an ID out of range; EDUP: an ID repeated or already free.  Checked
   before any change: on error nothing is freed. */
int flowkv_free(flowkv_allocator* a, const int32_t* ids, int32_t n);

/* Mark ids[0 .. n) in use without allocating them (blocks already held by
   resident requests).  ERANGE / EDUP as for flowkv_free, EDUP also for a block
   already in use.  On error nothing changes. */
int flowkv_mark_used(flowkv_allocator* a, const int32_t* ids, int32_t n);

/* Current free-space summary. */
int flowkv_allocator_stats(const flowkv_allocator* a, flowkv_alloc_stats* out);

/* ---- bidirectional segment alignment (section 3.3; Figure 3 caption) ------- */

/* Align one request: src_ids and dst_ids (n_blocks each, host memory) are the
   sender's and the receiver's block lists in logical order.  Writes the
   maximal runs with src and dst both stepping by +1 to out[0 .. *n_out), in
   logical order, `first` counting from 0.
   ERANGE: an ID outside its pool; EDUP: an ID repeated within src_ids or
   within dst_ids; ECAP: more than `cap` runs (*n_out = runs needed, out
   untouched);
   EINVAL: NULL pointers (arrays may be NULL when n_blocks == 0), negative
   sizes.  The run count is at most n_blocks. */
int flowkv_plan(const int32_t* src_ids, const int32_t* dst_ids, int32_t n_blocks,
                int32_t src_pool_blocks, int32_t dst_pool_blocks,
                flowkv_segment* out, int64_t cap, int64_t* n_out);

/* Align a batch of n_req requests in one call.  Request r's lists are
   src_ids[offsets[r] .. offsets[r+1]) and the same range of dst_ids; offsets
   has n_req + 1 non-decreasing entries starting at 0, and offsets[n_req] must
   fit int32.  Runs never cross requests; `first` runs across the whole batch.
   Receiver IDs must be distinct across the whole batch (one writer per
   block); sender IDs must be distinct within a request but may repeat across
   requests (shared prefix blocks).  Errors as for flowkv_plan. */
int flowkv_plan_batch(int32_t n_req, const int64_t* offsets,
                      const int32_t* src_ids, const int32_t* dst_ids,
                      int32_t src_pool_blocks, int32_t dst_pool_blocks,
                      flowkv_segment* out, int64_t cap, int64_t* n_out);

/* ---- transfer (section 3.3, Eq. 5 layouts; one launch for the whole plan) --- */

/* Enqueue one kernel on `hip_stream` (a hipStream_t; NULL = default stream)
   that copies, for every run in segs_dev[0 .. n_segs) and every layer and K/V,
   the run's blocks from `src` to `dst`.  segs_dev is device memory holding a
   plan made by flowkv_plan/flowkv_plan_batch for pools of these sizes;
   total_blocks is the plan's block count (last record's first + n_blocks).
   It is an argument because the launch is sized by it (a fixed number of
   tiles per block) before any record is read, and the records are in
   device memory, which the host could read back only with a synchronising
   copy; the caller holds the host plan it came from.
   The caller keeps segs_dev and both pools alive until the stream passes the
   kernel.  Asynchronous: returns once the launch is enqueued.  n_segs == 0 or
   total_blocks == 0 is a no-op.
   The kernel checks every run against both pools and skips, never touches
   outside the pools for, runs that fail the check.
   EINVAL: NULL pointers, pools that disagree on num_layers or chunk_bytes,
   bad layout, num_layers outside 1..FLOWKV_MAX_LAYERS, chunk_bytes not a
   positive multiple of 16, a base pointer not 16-byte aligned, a block of
   2 GiB or more, or src and dst memory ranges that overlap.
   EHIP: the runtime rejected the launch (message in flowkv_last_error()). */
int flowkv_transfer(const flowkv_pool* src, const flowkv_pool* dst,
                    const flowkv_segment* segs_dev, int64_t n_segs,
                    int64_t total_blocks, void* hip_stream);

/* flowkv_transfer with an explicit launch shape (cfg may be NULL = default).
   Same result for every valid shape; EINVAL for a shape outside the limits
   documented at flowkv_launch_config. */
int flowkv_transfer_ex(const flowkv_pool* src, const flowkv_pool* dst,
                       const flowkv_segment* segs_dev, int64_t n_segs,
                       int64_t total_blocks, const flowkv_launch_config* cfg,
                       void* hip_stream);

/* flowkv_transfer_ex for small plans held in host memory: the records are
   copied into the kernel's arguments at launch, so the plan needs no device
   buffer and no separate host-to-device copy; segs_host may be reused as
   soon as the call returns.  Same result as flowkv_transfer_ex with the same
   plan in device memory.  Up to FLOWKV_INLINE_RUNS records fit.  A plan in
   the planner's form (record i starts where record i - 1 ends, every record
   holds a block, and they cover [0, total_blocks)) travels as 12-byte
   records whose lengths follow from the next `first`, so more fit: up to
   FLOWKV_INLINE_RUNS_BLOCK_MAJOR between two block-major pools (one base
   pointer per side), and up to FLOWKV_INLINE_RUNS_LAYER_MAJOR when either
   pool is layer-major and the pools have at most FLOWKV_INLINE_LAYERS
   layers (one base pointer per layer and side); flowkv_inline_capacity
   gives the figure for two pools.  ECAP otherwise (use flowkv_transfer_ex
   with a device plan); other arguments and errors as for
   flowkv_transfer_ex. */
int flowkv_transfer_inline(const flowkv_pool* src, const flowkv_pool* dst,
                           const flowkv_segment* segs_host, int64_t n_segs,
                           int64_t total_blocks, const flowkv_launch_config* cfg,
                           void* hip_stream);

/* The most records of a planner-form plan (as flowkv_plan writes them) that
   flowkv_transfer_inline carries between pools src and dst:
   FLOWKV_INLINE_RUNS_BLOCK_MAJOR between two block-major pools, else
   FLOWKV_INLINE_RUNS_LAYER_MAJOR when neither pool has more than
   FLOWKV_INLINE_LAYERS layers, else FLOWKV_INLINE_RUNS.  Host only, no GPU
   call.  EINVAL for NULL arguments, an unknown layout or num_layers outside
   1..FLOWKV_MAX_LAYERS (*runs untouched). */
int flowkv_inline_capacity(const flowkv_pool* src, const flowkv_pool* dst, int64_t* runs);

/* Move one request (section 3.1's problem statement: K and V of request R
   from the sender's pool to the receiver's) in one call: flowkv_plan of src_ids
   and dst_ids (n_blocks each, host memory, pool sizes taken from the pool
   descriptors), then flowkv_transfer_inline with that plan.  *n_runs
   receives the plan's run count.  ECAP, with *n_runs set and nothing
   launched, when the plan has more runs than flowkv_transfer_inline carries
   between these pools (flowkv_inline_capacity; then plan with flowkv_plan
   and launch with a device plan).  Errors of the planner (ERANGE, EDUP) come before any launch; the
   others are flowkv_transfer_inline's.  n_blocks == 0 is a no-op. */
int flowkv_transfer_request(const flowkv_pool* src, const flowkv_pool* dst,
                            const int32_t* src_ids, const int32_t* dst_ids, int32_t n_blocks,
                            const flowkv_launch_config* cfg, int64_t* n_runs,
                            void* hip_stream);

/* Layer-wise variant (section 4.4 and Table 3: the "FlowKV-Layerwise"
   ablation, which moves the KV cache one layer at a time, as a sender that
   streams layers while prefill still runs would).  Moves only layers
   [layer_begin, layer_begin + layer_count) -- K and V -- of every run; other
   layers of the receiver's blocks are left unchanged.  Calling it for every
   layer, one launch each, gives the same bytes as one flowkv_transfer_ex.
   layer_count == 0 is a no-op.  EINVAL additionally for a layer range outside
   the pools; otherwise arguments and errors as for flowkv_transfer_ex. */
int flowkv_transfer_layers(const flowkv_pool* src, const flowkv_pool* dst,
                           const flowkv_segment* segs_dev, int64_t n_segs,
                           int64_t total_blocks, int32_t layer_begin, int32_t layer_count,
                           const flowkv_launch_config* cfg, void* hip_stream);

/* ---- decode attention over a pool (section 3.3: the PagedAttention kernel
        adapted to the restructured layout; the decode step of Eq. 2) -------- */

#define FLOWKV_ATTN_MAX_SPLIT 1024     /* most tokens per pass-1 workgroup    */
#define FLOWKV_ATTN_MIN_AUTO_SPLIT 256 /* least tokens the default rule picks */
#define FLOWKV_ATTN_AUTO_PAIRS 512     /* (request, split) pairs it aims at   */
#define FLOWKV_ATTN_INLINE_LENS 512    /* most host lengths a call carries in
                                          the kernel arguments               */

/* The split length used when split_tokens is 0: the smallest power of two s
   from FLOWKV_ATTN_MIN_AUTO_SPLIT to FLOWKV_ATTN_MAX_SPLIT with
   n_req x ceil(max_seq_len / s) <= FLOWKV_ATTN_AUTO_PAIRS, else
   FLOWKV_ATTN_MAX_SPLIT.  (Long splits amortise each workgroup's start-up
   and keep the merge small; a long request still gets tens of splits per
   KV head.)
   Writes it to *split_tokens.  EINVAL for a NULL output or negative sizes. */
int flowkv_decode_attention_split(int32_t n_req, int32_t max_seq_len, int32_t* split_tokens);

/* Workspace bytes flowkv_decode_attention needs for n_req requests of at most
   max_seq_len tokens: n_req x q_heads x ceil(max_seq_len / split_tokens) x
   (head_dim + 2) floats, split_tokens 0 meaning the default rule above. */
int flowkv_decode_attention_workspace(int32_t n_req, int32_t q_heads, int32_t head_dim,
                                      int32_t max_seq_len, int32_t split_tokens,
                                      int64_t* bytes);

/* One decode step of attention for n_req requests, layer `layer` of a bf16
   pool (either layout; the pool's chunk_bytes must be block_size x kv_heads x
   head_dim x 2).  For request r and query head h (KV head g = h / (q_heads /
   kv_heads)), with T = seq_lens[r] tokens in blocks block_tables[r][0..]:
       out[r][h] = sum_t softmax_t(scale * q[r][h] . K[t][g]) * V[t][g]
   Token t lives in block block_tables[r * max_blocks + t / block_size], slot
   t % block_size.  Device inputs: q (n_req, q_heads, head_dim) bf16, 16-byte
   aligned; block_tables (n_req, max_blocks) int32; seq_lens_dev (n_req)
   int32.  seq_lens_host: the same lengths in host memory, or NULL.  When it
   is given and n_req <= FLOWKV_ATTN_INLINE_LENS, the lengths travel in the
   kernel arguments (copied at the call; the array may be reused as soon as
   it returns) and seq_lens_dev is not read and may be NULL: a split past its
   request's end then costs no memory access, which speeds up batches of
   mixed lengths.  The two copies must agree; the host copy decides.
   Output: out (n_req, q_heads, head_dim) float32.  workspace: device memory
   of at least flowkv_decode_attention_workspace(...) bytes, owned by the
   caller, busy until the stream passes the call (NULL when that is 0).  Tokens beyond
   max_blocks x block_size or beyond max_seq_len are not read; a block ID
   outside the pool contributes nothing; a request with no tokens gets zeros.
   head_dim 64 or 128; q_heads / kv_heads in {1, 2, 4, 8}; split_tokens 0 =
   the default rule (flowkv_decode_attention_split), else
   1..FLOWKV_ATTN_MAX_SPLIT.  Two launches on hip_stream.  At most 65,535
   requests and 65,535 splits (ceil(max_seq_len / split_tokens)) per call,
   and max_blocks x block_size at most 2^31 - 1 tokens.
   EINVAL for bad shapes or pointers, ECAP for a short workspace. */
int flowkv_decode_attention(const flowkv_pool* pool, int32_t layer, const void* q_dev,
                            int32_t n_req, int32_t q_heads, int32_t kv_heads,
                            int32_t head_dim, const int32_t* block_tables_dev,
                            int32_t max_blocks, const int32_t* seq_lens_dev,
                            const int32_t* seq_lens_host, int32_t max_seq_len, float scale,
                            int32_t split_tokens, float* out_dev, void* workspace_dev,
                            int64_t workspace_bytes, void* hip_stream);

/* For callers that cannot allocate device memory or pass a workspace: code
   under HIP graph capture, serving loops and harnesses that forbid
   hipMalloc.  flowkv_decode_attention with the workspace replaced by
   FLOWKV_ATTN_SCRATCH_BYTES of device memory the library holds on each GPU it
   runs on, from the first call on that GPU until the process ends.  The call
   allocates nothing (no hipMalloc, hipFree or allocating library routine);
   the first call on a GPU looks up that GPU's copy of the array
   (hipGetSymbolAddress) with the GPU current.  The caller still passes q,
   the block tables, the lengths and the output, as for
   flowkv_decode_attention, with the same results for the same inputs.
   ECAP, with nothing launched, when the call needs more partial results
   than the scratch holds: flowkv_decode_attention_workspace(...) above
   FLOWKV_ATTN_SCRATCH_BYTES (16 MiB covers, for example, 32 requests of up
   to 20,480 tokens with 32 query heads of head_dim 128 at the default
   split).  Calls on one GPU share its scratch: calls that overlap on that
   GPU (other streams, other threads) race and give undefined results;
   serialise them.  Other arguments and errors as for
   flowkv_decode_attention. */
#define FLOWKV_ATTN_SCRATCH_BYTES 16777216 /* 16 MiB */

int flowkv_decode_attention_noalloc(const flowkv_pool* pool, int32_t layer, const void* q_dev,
                                    int32_t n_req, int32_t q_heads, int32_t kv_heads,
                                    int32_t head_dim, const int32_t* block_tables_dev,
                                    int32_t max_blocks, const int32_t* seq_lens_dev,
                                    const int32_t* seq_lens_host, int32_t max_seq_len,
                                    float scale, int32_t split_tokens, float* out_dev,
                                    void* hip_stream);

/* ---- load-aware scheduler (section 3.4; Appendix A, Algorithm 1) ------------
   Host only.  Each node reports a status vector S_i of 12 indicators, in
   Algorithm 1's order:
     0 L_r^p  1 L_w^p  2 L_sw^p  3 L_se^p   running, waiting, swapped and sending
     4 L_r^d  5 L_w^d  6 L_sw^d  7 L_se^d   queue lengths, prefill then decode
     8 T_b    9 KV_u  10 G_u    11 MB_u     token budget, KV-cache, GPU and
                                            memory-bandwidth utilisation
   The scheduler keeps a sliding window of samples per node; an evaluation
   takes the window mean of each indicator divided by its scale, forms
       C_i^p = w_p . (L_r^p, L_w^p, L_sw^p, L_se^p, T_b, KV_u, G_u, MB_u)
       C_i^d = w_d . (L_r^d, L_w^d, L_sw^d, L_se^d, T_b, KV_u, G_u, MB_u)
   (term by term in that order), averages C_i^p over the prefill-role nodes
   and C_i^d over the decode-role nodes (0 for a role with no node), and
   picks the scenario, testing in this order: low load when |C^p| < eps_p_min
   and |C^d| < eps_d_min; normal when |C^p| <= eps_p_low and |C^d| <=
   eps_d_low; imbalanced when both are within the high thresholds; extreme
   (overload) otherwise.  Offline nodes (FLOWKV_ROLE_OFFLINE) report status
   but count in no average, no idle set and no route.
   Readings of what Algorithm 1 leaves open:
     - idle nodes (imbalanced) are the nodes of the less loaded role whose
       own-role score is below idle_threshold; they are to take the busier
       role, the one with the larger C / eps_low;
     - extreme load asks for one more node of each role whose |C| exceeds
       its high threshold once the scenario has lasted scale_after
       consecutive evaluations (the count restarts after each scale request
       and after any other scenario);
     - low load is the other extreme scenario section 3.4 names (Appendix
       A: scale up or, conversely, down once the scores have lasted);
       Algorithm 1's branches would read it as normal, so it is tested
       first, against a lower pair of thresholds (0 = never).  Once it has
       lasted scale_after consecutive evaluations, each role with more than
       one node may give one up (scale_* = -1), with its own count;
     - routing (flowkv_sched_route) takes the prefill node with the least
       (queued tokens + prompt tokens not in its prefix cache) / prefill
       rate, then the decode node with room for the KV bytes and the least
       latency + bytes x seconds-per-byte from that prefill node; ties go
       to the lower index.
   All arithmetic is IEEE double in the order stated, so results are exact
   functions of the inputs.  Handles are not thread-safe. */

#define FLOWKV_SCHED_INDICATORS 12
#define FLOWKV_SCHED_TERMS 8
#define FLOWKV_SCHED_MAX_WINDOW 4096

enum { FLOWKV_ROLE_PREFILL = 0, FLOWKV_ROLE_DECODE = 1, FLOWKV_ROLE_OFFLINE = 2 };
enum {
  FLOWKV_SCENARIO_NORMAL = 0,
  FLOWKV_SCENARIO_IMBALANCED = 1,
  FLOWKV_SCENARIO_EXTREME = 2,  /* overload */
  FLOWKV_SCENARIO_LOW_LOAD = 3  /* the extreme scenario's low-load side */
};

typedef struct flowkv_sched_params {
  int32_t window;       /* samples in the sliding window, 1..FLOWKV_SCHED_MAX_WINDOW */
  int32_t scale_after;  /* consecutive extreme evaluations before a scale request, >= 1 */
  double scale[FLOWKV_SCHED_INDICATORS];  /* normalisation divisors, > 0 */
  double w_prefill[FLOWKV_SCHED_TERMS];   /* w_r, w_w, w_sw, w_se, w_t, w_kv, w_g, w_mb */
  double w_decode[FLOWKV_SCHED_TERMS];
  double eps_p_low, eps_d_low;            /* > 0 */
  double eps_p_high, eps_d_high;          /* >= the low thresholds */
  double idle_threshold;
  double eps_p_min, eps_d_min;            /* low load below both; 0 <= min <= low */
} flowkv_sched_params;

typedef struct flowkv_sched_result {
  int32_t scenario;       /* FLOWKV_SCENARIO_* */
  int32_t n_idle;         /* idle node indices written (imbalanced), else 0 */
  int32_t switch_to;      /* the role idle nodes take (imbalanced), else -1 */
  int32_t scale_prefill;  /* +1: add a prefill node (overload, persisted);
                             -1: one may go offline (low load, persisted) */
  int32_t scale_decode;   /* the same for the decode role */
  int32_t reserved;
  double c_prefill;       /* C^p */
  double c_decode;        /* C^d */
} flowkv_sched_result;

typedef struct flowkv_sched flowkv_sched; /* opaque, host memory only */

/* New scheduler for n_nodes nodes (1..2^20) with initial roles[n_nodes]
   (FLOWKV_ROLE_*, offline included).  The parameters are copied.  EINVAL for bad parameters,
   ENOSPC if host memory runs out. */
int flowkv_sched_create(const flowkv_sched_params* params, int32_t n_nodes,
                        const int32_t* roles, flowkv_sched** out);
void flowkv_sched_destroy(flowkv_sched* s);

/* Change one node's role (a hybrid node switching, a node going offline
   after a scale-down, or an offline node joining after a scale-up). */
int flowkv_sched_set_role(flowkv_sched* s, int32_t node, int32_t role);

/* One sample of every node's status: status[n_nodes x 12], row-major. */
int flowkv_sched_observe(flowkv_sched* s, const double* status);

/* One evaluation of Algorithm 1 over the samples in the window.  Writes
   *res; idle node indices, ascending, to idle_nodes[0 .. res->n_idle)
   (room for n_nodes; may be NULL only if the caller ignores them: then
   n_idle is still set); node_scores[n_nodes x 2] = (C_i^p, C_i^d) if not
   NULL.  EINVAL before the first observation. */
int flowkv_sched_evaluate(flowkv_sched* s, flowkv_sched_result* res, int32_t* idle_nodes,
                          double* node_scores);

/* Routing of one request (normal load; the same rule serves the other
   scenarios).  Per node i (all arrays n_nodes long; only the current role
   is looked at): prefix_hit[i] prompt tokens already cached on i,
   queued_tokens[i] prefill tokens waiting on i, prefill_rate[i] tokens per
   second (nodes with rate <= 0 are skipped), free_bytes[i] KV bytes the node
   can receive; xfer_sec_per_byte and xfer_latency are n_nodes x n_nodes,
   row = sender.  Writes the chosen nodes, -1 where none qualifies. */
int flowkv_sched_route(const flowkv_sched* s, int64_t prompt_tokens, const int64_t* prefix_hit,
                       const int64_t* queued_tokens, const double* prefill_rate,
                       int64_t kv_bytes, const double* xfer_sec_per_byte,
                       const double* xfer_latency, const int64_t* free_bytes,
                       int32_t* prefill_node, int32_t* decode_node);

/* ---- diagnostics ------------------------------------------------------------ */

/* Static name of a status code. */
const char* flowkv_strerror(int code);

/* The calling thread's most recent error message ("" if none). */
const char* flowkv_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FLOWKV_H */
