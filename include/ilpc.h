/*
 * ilpc.h -- C ABI of the prefix-cached paged prefill attention library
 * (libilpc.so) for AMD Instinct MI355X (gfx950).
 *
 * The operations are the hot path of LLM-based online log parsing with
 * prefix caching, as described by InferLog (arXiv 2507.08523):
 *   - a prompt is an instruction, k demonstrations and the queried log
 *     (section 2.1.1, prompt format);
 *   - KV of a shared prompt prefix is reused across requests at block
 *     granularity, and a block is reusable only if every block before it is
 *     reused too (section 2.1.2 on the KV cache and prefix caching, and
 *     its three-request figure);
 *   - the KV of cache-missing tokens is computed and stored (section 3.2.2);
 *   - prefill over the uncached suffix against cached + new KV dominates the
 *     latency (section 2.2.1).
 *
 * Conventions for every call:
 *   - Return value: ILPC_OK (0) or a negative ILPC_E* code.  No exception or
 *     abort crosses the ABI.  ilpc_last_error() gives a message for the last
 *     failing call on the calling thread.
 *   - Arguments are validated before any state change or kernel launch.  A
 *     failing call leaves the cache unchanged; its outputs are unspecified.
 *   - Host pointers are marked [host], device pointers [device].  The caller
 *     owns every buffer (including the attention workspace); the library owns
 *     the cache and ICL-table handles (host memory) and one static device
 *     array (the scratch of ilpc_paged_prefill_attn_noalloc), and allocates
 *     no device memory.
 *   - bf16 tensors are passed as uint16_t* holding the raw bf16 bits.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Device calls are
 *     asynchronous on that stream; they return ILPC_EHIP when the launch
 *     fails.  Work ordered on one stream needs no other synchronisation.
 *   - Supported shapes: block_size == 16, head_dim in {64, 128},
 *     Hq % Hkv == 0, 1 <= Hq / Hkv <= 64.  Anything else is ILPC_EUNSUP.
 *
 * Device layouts (row-major, bf16):
 *   k_pool [num_blocks, Hkv, 16, D]  key rows of a block, token-major
 *   v_pool [num_blocks, Hkv, D, 16]  value rows of a block, transposed
 *                                    (dimension-major), the operand layout
 *                                    the matrix cores consume directly
 *   q, out [total_q, Hq, D]          packed query / output rows
 *   k_new, v_new [total_new, Hkv, D] packed rows to append
 *   block_tables [B, max_blocks] int32, physical block of each logical
 *                                    block of a request, -1 past the end
 */
#ifndef ILPC_H
#define ILPC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  ILPC_OK = 0,
  ILPC_EINVAL = -1, /* bad argument (null pointer, negative size, bad lengths) */
  ILPC_ENOSPC = -2, /* the block pool cannot hold the batch's new blocks */
  ILPC_ETABLE = -3, /* the block-key table cannot hold the batch's new keys */
  ILPC_EUNSUP = -4, /* shape outside the supported set */
  ILPC_EHIP = -5    /* a HIP runtime call or kernel launch failed */
};

/* ilpc_prefix_match flags */
#define ILPC_NO_LOOKUP 1u   /* ignore the table: every request has P = 0 */
#define ILPC_NO_REGISTER 2u /* do not register the batch's new full blocks */

typedef struct ilpc_cache ilpc_cache; /* opaque, host memory, library-owned */

/* Message describing the last non-OK return on this thread ("" if none).
 * The pointer stays valid until the next failing call on the same thread. */
const char* ilpc_last_error(void);

/* Create an empty prefix cache over a pool of `num_blocks` physical blocks of
 * `block_size` tokens (must be 16).  The block-key table has
 * 2^table_log2_cap slots (1 <= table_log2_cap <= 30) and holds at most
 * 7/8 of that many keys.  *out receives the handle. */
int ilpc_cache_create(int32_t num_blocks, int32_t block_size, int32_t table_log2_cap,
                      ilpc_cache** out);

/* Free a cache (NULL is ignored). */
void ilpc_cache_destroy(ilpc_cache* cache);

/* Forget every registered block and restart the block allocator at 0. */
int ilpc_cache_reset(ilpc_cache* cache);

/* stats[0] = registered keys, stats[1] = next free block id (for an LRU
 * cache: blocks not on the free queue), stats[2] = key capacity (7/8 of the
 * slots), stats[3] = num_blocks. */
int ilpc_cache_stats(const ilpc_cache* cache, int64_t stats[4]);

/* Record the current state so that ilpc_cache_rollback can return to it:
 * mark[0] = registered-key journal length, mark[1] = next free block id.
 * ILPC_EUNSUP on an LRU cache (as is ilpc_cache_rollback). */
int ilpc_cache_checkpoint(const ilpc_cache* cache, int64_t mark[2]);

/* Undo every registration and block allocation made since `mark` was taken
 * (most recent first).  A mark from before a later reset or rollback past it
 * is rejected with ILPC_EINVAL. */
int ilpc_cache_rollback(ilpc_cache* cache, const int64_t mark[2]);

/*
 * A prefix cache whose blocks have a lifecycle (section 2.1.2: KV blocks live
 * in bounded GPU memory and are evicted least recently used first).  Matching
 * and registration are those of ilpc_prefix_match; what differs is where
 * block ids come from and when they return.  A block is
 *   in use   -- held by at least one request not yet released (count > 0);
 *   cached   -- held by none but its key still registered: a later request
 *               can hit it; these blocks form the LRU list;
 *   free     -- held by none and named by no key; on the free queue, which
 *               starts as 0, 1, ..., num_blocks-1.
 * ilpc_prefix_match on such a cache first pins every block the batch hits (in
 * request order), then takes each new block from the front of the free queue,
 * or, when the queue is empty, the head of the LRU list (least recently used),
 * whose key is removed from the table.  It returns ILPC_ENOSPC, changing
 * nothing, when the batch needs more new blocks than the free blocks plus the
 * cached blocks it does not hit.  Without releases, ids come out exactly as
 * from ilpc_cache_create's bump allocator.  The key capacity
 * (7/8 * 2^table_log2_cap) must be >= num_blocks (ILPC_EINVAL otherwise), so
 * ILPC_ETABLE never occurs.  Host memory only; the device pools are the
 * caller's and are not touched.
 */
int ilpc_cache_create_lru(int32_t num_blocks, int32_t block_size, int32_t table_log2_cap,
                          ilpc_cache** out);

/*
 * Requests finished: drop one hold on every block of each row of
 * block_tables [host] int32 [B, max_blocks] (a row ends at its first -1), the
 * rows as ilpc_prefix_match returned them.  Each row is released from its
 * last block to its first; a block whose count reaches 0 goes to the tail of
 * the LRU list if its key is registered, else to the back of the free queue
 * (so a cached prompt loses its end before its start).  ILPC_EINVAL, changing
 * nothing, if an id is out of range or a block would be released more often
 * than it is held; ILPC_EUNSUP on a cache from ilpc_cache_create.
 */
int ilpc_cache_release(ilpc_cache* cache, const int32_t* block_tables, int32_t B,
                       int32_t max_blocks);

/* Mark cached blocks as just used: each id of block_ids [host] int32 [n] that
 * names a cached block moves to the LRU tail, in order; ids of blocks in use
 * or free, and -1 entries, change nothing.  ILPC_EINVAL (nothing changed) for
 * an id outside [0, num_blocks) other than -1. */
int ilpc_cache_touch(ilpc_cache* cache, const int32_t* block_ids, int32_t n);

/* usage[0] = blocks in use, usage[1] = cached blocks, usage[2] = free blocks,
 * usage[3] = evictions so far.  For a cache from ilpc_cache_create every
 * allocated block counts as in use. */
int ilpc_cache_usage(const ilpc_cache* cache, int64_t usage[4]);

/* The cached blocks, least recently used first: writes min(max_ids, count)
 * ids to block_ids [host] int32 [max_ids] and the count to *n_cached. */
int ilpc_cache_lru_order(const ilpc_cache* cache, int32_t* block_ids, int32_t max_ids,
                         int32_t* n_cached);

/*
 * Block-level prefix matching of one batch (section 2.1.2).
 *
 * tokens      [host] int32 [cu_seqlens[B]]  the prompts, packed
 * cu_seqlens  [host] int32 [B+1]            prompt r is tokens[cu[r]..cu[r+1]),
 *                                           cu[0] = 0, every length >= 1
 * B           number of prompts (0 is a no-op)
 * reserve     [host] int32 [B] or NULL      extra tokens (later decode steps)
 *                                           to allocate blocks for
 * max_blocks  row length of block_tables; must be >= ceil((L_r+reserve_r)/16)
 * flags       ILPC_NO_LOOKUP | ILPC_NO_REGISTER
 * cached_len  [host] int32 [B]              out: P_r, a multiple of 16
 * block_tables [host] int32 [B*max_blocks]  out: physical block ids, -1 pad
 * block_keys  [host] uint64 [B*max_blocks] or NULL  out: chained key of each
 *                                           full block, 0 past them
 *
 * Every full 16-token block b of prompt r gets the chained key
 *   c_b = fmix64(c_{b-1} XOR d_b),  c_{-1} = 0x243F6A8885A308D3,
 *   d_b = fmix64(sum_i fmix64(w_i XOR (i+1)*0x9E3779B97F4A7C15)), i = 0..7,
 *   w_i = u32(t_{2i}) | u32(t_{2i+1}) << 32 over the block's tokens,
 * with fmix64 the MurmurHash3 finaliser and a key of 0 replaced by 1.
 * All prompts are matched against the table as it stood before the call
 * (frozen snapshot): P_r = 16 * (length of the longest run of leading keys
 * present), capped at floor((L_r - 1) / 16) blocks so that at least one token
 * is recomputed.  Cached blocks reuse their registered ids; every other block
 * of the prompt (and of its reserve) gets the next id of a bump allocator,
 * prompt by prompt.  Afterwards the new full blocks are registered in prompt
 * order, first registration winning.  ILPC_ENOSPC if ids would exceed
 * num_blocks; ILPC_ETABLE if held keys + new full blocks would exceed the key
 * capacity.  Synchronous, host only.
 */
int ilpc_prefix_match(ilpc_cache* cache, const int32_t* tokens, const int32_t* cu_seqlens,
                      int32_t B, const int32_t* reserve, int32_t max_blocks, uint32_t flags,
                      int32_t* cached_len, int32_t* block_tables, uint64_t* block_keys);

/*
 * Store the K/V of cache-missing tokens into the paged pools (section 3.2.2).
 *
 * k_new, v_new [device] bf16 [cu_new[B], Hkv, D]
 * k_pool       [device] bf16 [num_blocks, Hkv, 16, D]
 * v_pool       [device] bf16 [num_blocks, Hkv, D, 16]
 * block_tables [device] int32 [B, max_blocks]
 * cu_new       [device] int32 [B+1]   rows of request r: cu_new[r]..cu_new[r+1]
 * start_pos    [device] int32 [B]     absolute position of request r's first row
 * max_new      [host]   upper bound of cu_new[r+1]-cu_new[r] over r
 *
 * Row t of request r is written to position p = start_pos[r] + t, i.e. to
 * logical block p/16, slot p%16.  Rows beyond max_new, and rows whose logical
 * block is >= max_blocks or maps to an id outside [0, num_blocks), are not
 * written (no out-of-bounds access is made).
 */
int ilpc_kv_append(const uint16_t* k_new, const uint16_t* v_new, uint16_t* k_pool,
                   uint16_t* v_pool, int32_t num_blocks, const int32_t* block_tables,
                   int32_t max_blocks, const int32_t* cu_new, const int32_t* start_pos, int32_t B,
                   int32_t max_new, int32_t Hkv, int32_t D, int32_t block_size, void* stream);

/*
 * Rotary position embedding fused into the K/V append (section 2.1.2: the
 * stored KV carries each token's position).  Same rows, pools, tables and
 * bounds rules as ilpc_kv_append, plus:
 *
 * q        [device] bf16 [cu_new[B], Hq, D] or NULL  query rows of the same
 *                   tokens (packed like k_new)
 * q_out    [device] bf16 [cu_new[B], Hq, D] or NULL  rotated queries; may be
 *                   q itself (in place); NULL exactly when q is NULL
 * inv_freq [device] fp32 [D/2]  angle per position of dimension pair i
 *                   (base^(-2i/D) for plain RoPE; any scaled variant the
 *                   model uses is the caller's table)
 *
 * Row t of request r sits at position p = start_pos[r] + t.  For i < D/2 the
 * pair (x_i, x_{i+D/2}) of its K row and of each of its Q rows becomes
 *   (x_i cos a - x_{i+D/2} sin a,  x_{i+D/2} cos a + x_i sin a),
 *   a = fl32(p * inv_freq[i]),
 * computed in fp32 from the bf16 inputs and rounded to bf16 (nearest even);
 * the rotated K row is stored in the pool, V unchanged.  Q rows are rotated
 * even where the block id is outside [0, num_blocks) (only K/V are skipped);
 * rows past max_new or whose logical block is >= max_blocks are not written.
 * Supported: D in {64, 128}, Hq % Hkv == 0, Hq / Hkv <= 64.
 */
int ilpc_rope_kv_append(const uint16_t* q, uint16_t* q_out, int32_t Hq, const uint16_t* k_new,
                        const uint16_t* v_new, uint16_t* k_pool, uint16_t* v_pool,
                        int32_t num_blocks, const int32_t* block_tables, int32_t max_blocks,
                        const int32_t* cu_new, const int32_t* start_pos, int32_t B,
                        int32_t max_new, int32_t Hkv, int32_t D, int32_t block_size,
                        const float* inv_freq, void* stream);

/*
 * Decode-shaped paged attention (section 2.1.2: each generated token attends
 * to the cached KV of its whole context): the same operation, arguments,
 * layouts and bounds rules as ilpc_paged_prefill_attn, for batches whose
 * max_q_len * (Hq / Hkv) <= 32 (ILPC_EUNSUP otherwise).  One wave per
 * (request, kv head) pair streams that request's K/V blocks from the pools;
 * results agree with ilpc_paged_prefill_attn to the attention tolerance, not
 * bit for bit.  ilpc_paged_prefill_attn takes this path by itself for such
 * batches: split as ilpc_decode_split() says when its workspace has room for
 * the partials, else unsplit when B * Hkv >= the device's compute units.
 *
 * n_split      [host] key ranges per pair, 1 .. 64, or 0 for
 *                     ilpc_decode_split()'s choice.  With n > 1 each range is
 *                     one wave; the ranges' partial results (fp32) go to the
 *                     workspace and a second kernel merges them, so that
 *                     batches with few pairs still occupy the whole chip.
 * workspace    [device] >= ilpc_decode_workspace_bytes(..., n) bytes,
 *                     16-byte aligned, no initial contents needed (NULL with
 *                     0 bytes when n = 1).  Calls that may run concurrently
 *                     need separate workspaces.
 * A short or misaligned workspace, or n_split outside [0, 64], is ILPC_EINVAL.
 */
int ilpc_paged_decode_attn(const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool,
                           int32_t num_blocks, const int32_t* block_tables, int32_t max_blocks,
                           const int32_t* cu_q, const int32_t* seq_lens, int32_t B, int32_t max_q_len,
                           int32_t Hq, int32_t Hkv, int32_t D, int32_t block_size, float softmax_scale,
                           uint16_t* out, int32_t n_split, void* workspace, size_t workspace_bytes,
                           void* stream);

/* The key-range count ilpc_paged_decode_attn uses for n_split = 0 on the
 * current device: 1 when B * Hkv >= its SIMDs (4 per compute unit), and
 * when B * Hkv >= half of them with a context bound 16 * max_blocks under
 * 1024 tokens; otherwise enough ranges for one wave per SIMD, at most one
 * per 32 keys of that bound, at most 64. */
int ilpc_decode_split(int32_t B, int32_t Hkv, int32_t max_blocks, int32_t* n_split);

/* Workspace bytes of ilpc_paged_decode_attn with n_split ranges:
 * 0 for n_split = 1, else B * Hkv * n_split * min(32, max_q_len * Hq / Hkv) * (D + 2) * 4. */
int ilpc_decode_workspace_bytes(int32_t B, int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D,
                                int32_t n_split, size_t* bytes);

/* Bytes of device workspace ilpc_paged_prefill_attn needs for these sizes:
 * 64 (the counters of its work queues), plus, for decode-shaped batches
 * (max_q_len * Hq / Hkv <= 32) with fewer (request, kv head) pairs than the
 * current device has SIMDs, room for the split decode kernel's partials
 * (ilpc_decode_workspace_bytes() at the split of any context length).  A
 * workspace of only 64 bytes is still accepted: such batches then run
 * unsplit. */
int ilpc_attn_workspace_bytes(int32_t B, int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D,
                              size_t* bytes);

/*
 * Causal grouped-query attention of each request's newest q_len_r tokens
 * over its whole context, read from the paged pools through the block table
 * (section 2.1.2 prefill with reused prefix KV; a decode step is q_len_r = 1).
 *
 * q            [device] bf16 [cu_q[B], Hq, D]
 * k_pool, v_pool as for ilpc_kv_append, already holding every context token
 * block_tables [device] int32 [B, max_blocks]
 * cu_q         [device] int32 [B+1]  query rows of request r: cu_q[r]..cu_q[r+1]
 * seq_lens     [device] int32 [B]    context length L_r (cached + new tokens)
 * max_q_len    [host]   >= every q_len_r; rows beyond it are not computed
 * softmax_scale         multiplies q.k before the softmax (1/sqrt(D) usually)
 * out          [device] bf16 [cu_q[B], Hq, D]
 * workspace    [device] >= 64 bytes (ilpc_attn_workspace_bytes() for every
 *                      path), 16-byte aligned, its first 64 bytes zero-filled
 *                      before the first use.  Each call leaves them zero-filled
 *                      again when its kernels complete (the rest is scratch),
 *                      so calls ordered on one stream can share it; calls that
 *                      may run concurrently (different streams) need separate
 *                      ones.
 *
 * Query t of request r sits at position L_r - q_len_r + t and attends to keys
 * 0 .. L_r - q_len_r + t; q head h reads kv head h / (Hq/Hkv).  Products and
 * sums in fp32 (matrix cores take bf16 operands), online softmax in fp32,
 * output rounded to bf16 (nearest-even).  A request with q_len_r > L_r, with
 * L_r > 16 * max_blocks, or whose blocks map outside [0, num_blocks) gets
 * unspecified output rows but causes no out-of-bounds access.  Block tables
 * wider than 2^24 blocks are ILPC_EUNSUP; a missing or short workspace is
 * ILPC_EINVAL.
 */
int ilpc_paged_prefill_attn(const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool,
                            int32_t num_blocks, const int32_t* block_tables, int32_t max_blocks,
                            const int32_t* cu_q, const int32_t* seq_lens, int32_t B,
                            int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D,
                            int32_t block_size, float softmax_scale, uint16_t* out,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * ilpc_paged_prefill_attn without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation).  It allocates nothing: its
 * workspace is a static device array of the library, 8 MiB + 256 bytes, one
 * per GPU, held from its first use on that GPU until the process ends.  The
 * first call on a device looks up that device's copy (with the device
 * current); later calls reuse the address.
 *
 * Arguments, layouts, bounds rules and the result are those of
 * ilpc_paged_prefill_attn with a workspace of 8 MiB + 256 bytes, and the
 * kernels are the same: the first 64 bytes hold the work-queue counters
 * (zero when the library is loaded; every call leaves them zero again), and
 * decode-shaped batches split their keys over several waves only when the
 * split's partial results fit in the rest (else they run unsplit), so no
 * batch needs more scratch than the array holds and none is refused for its
 * size.  Every call on a GPU shares that GPU's array: calls that may overlap
 * on one GPU (different streams, other threads) race and must not be issued;
 * calls ordered on one stream are safe.  ILPC_EHIP if the array's address
 * cannot be looked up on the current device.
 */
int ilpc_paged_prefill_attn_noalloc(const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool,
                                    int32_t num_blocks, const int32_t* block_tables, int32_t max_blocks,
                                    const int32_t* cu_q, const int32_t* seq_lens, int32_t B,
                                    int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D,
                                    int32_t block_size, float softmax_scale, uint16_t* out, void* stream);

/* Bytes of device workspace ilpc_paged_prefill_attn_cascade needs:
 * 256 + align256(B*max_q_len*Hq*D*4) + align256(B*max_q_len*Hq*8). */
int ilpc_attn_cascade_workspace_bytes(int32_t B, int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D,
                                      size_t* bytes);

/*
 * The same attention as ilpc_paged_prefill_attn, split at a prefix that every
 * request of the batch shares (the instruction and leading demonstrations of
 * the log-parsing prompts, section 2.1.1, which prefix caching stores once,
 * section 2.1.2): the shared keys are read once per 256 query columns of the
 * whole batch (query row x q head of a kv head), not once per request.
 *   - Prefill-shaped batches (max_q_len * Hq / Hkv >= 64) whose shared prefix
 *     holds at least three 64-key tiles, and whose per-item tile list fits
 *     ((256 / G + 1) * (ceil(16 * max_blocks / 64) - floor(shared_len / 64))
 *     <= 2048, G = Hq / Hkv), run as one launch: each workgroup takes 256
 *     columns of the batch, attends them to the floor(shared_len / 64) * 64
 *     shared keys, then to each of their requests' own keys from there on
 *     (masked to that request's columns, causal), in one online softmax.
 *   - Other batches (decode steps among them) run two launches: every query
 *     row over keys 0 .. shared_len-1, with the unnormalised state in the
 *     workspace, then each request's queries over its keys shared_len ..
 *     L_r-1, continuing from that state.
 *
 * shared_len  [host] a multiple of 16 in [0, 16*max_blocks].  The caller
 *             guarantees that the first shared_len/16 entries of every
 *             request's block table equal request 0's, and that shared_len <=
 *             L_r - q_len_r for every request (the shared keys precede every
 *             query).  0 runs ilpc_paged_prefill_attn's single pass.
 * workspace   [device] >= ilpc_attn_cascade_workspace_bytes() bytes,
 *             16-byte aligned, its first 128 bytes zero-filled before the
 *             first use (each call leaves them zero-filled again); the rest
 *             holds fp32 partial results of the two-launch form,
 *             overwritten by every such call.
 * Other arguments and the result as for ilpc_paged_prefill_attn; rows of
 * requests whose q_len exceeds max_q_len are not computed.  If the
 * shared_len contract does not hold the output is unspecified, but no
 * out-of-bounds access is made.  Results agree with the single pass within
 * rounding (the summation order differs).
 */
int ilpc_paged_prefill_attn_cascade(const uint16_t* q, const uint16_t* k_pool, const uint16_t* v_pool,
                                    int32_t num_blocks, const int32_t* block_tables, int32_t max_blocks,
                                    const int32_t* cu_q, const int32_t* seq_lens, int32_t B,
                                    int32_t max_q_len, int32_t Hq, int32_t Hkv, int32_t D,
                                    int32_t block_size, int32_t shared_len, float softmax_scale,
                                    uint16_t* out, void* workspace, size_t workspace_bytes, void* stream);

/*
 * Scheduler steps of a chunked prefill (the per-step token bound that section
 * 3.3 tunes, vLLM's max-num-batched-tokens; section 4.1's PC-Chunk baseline).
 * Host only.
 *
 * q_lens      [host] int32 [B]  new (uncached) tokens of each request, >= 0
 * budget      new tokens per step, >= 1
 * max_pieces  room of the four piece arrays
 * piece_req, piece_off, piece_len, piece_step  [host] int32 [max_pieces]
 *             out: piece k is tokens piece_off[k] .. piece_off[k] +
 *             piece_len[k] - 1 of request piece_req[k]'s new tokens, run in
 *             step piece_step[k]
 * n_pieces, n_steps  out: the number of pieces and of steps (also set when
 *             the pieces do not fit, so a call with max_pieces = 0 sizes them)
 *
 * First come, first served over the requests in order: a step takes what is
 * left of the current request, then the following ones, and cuts the last
 * one it reaches, so every step but the last holds exactly `budget` tokens
 * and a step is a contiguous run of the batch's packed new-token rows.
 * Pieces come in step order and, within a step, request order; requests with
 * no new tokens get none.  ILPC_EINVAL for a negative length, budget < 1, or
 * pieces that do not fit in max_pieces.
 */
int ilpc_chunk_schedule(const int32_t* q_lens, int32_t B, int32_t budget, int32_t max_pieces,
                        int32_t* piece_req, int32_t* piece_off, int32_t* piece_len, int32_t* piece_step,
                        int32_t* n_pieces, int32_t* n_steps);

/*
 * Split point for ilpc_paged_prefill_attn_cascade: the keys at the front that
 * every request of the batch shares (the instruction and leading
 * demonstrations, section 2.1.1, stored once by the prefix cache, section
 * 2.1.2).  Host only.
 *
 * cached_len   [host] int32 [B]              P_r of each request, >= 0
 * block_tables [host] int32 [B, max_blocks]  as ilpc_prefix_match returned them
 * shared_len   out: 16 * the longest run of leading block ids that are equal
 *              (and >= 0) in every row, capped at floor(min_r P_r / 16)
 *              blocks, so that the shared keys precede every query; 0 for B = 0.
 */
int ilpc_shared_prefix_len(const int32_t* cached_len, const int32_t* block_tables, int32_t B,
                           int32_t max_blocks, int32_t* shared_len);

/*
 * Whether ilpc_paged_prefill_attn_cascade at shared_len is the faster choice
 * for this batch than ilpc_paged_prefill_attn (host only).  The split does
 * the same matrix-core work (section 2.1.2: every query still meets every
 * key); in one launch it reads the shared K/V once per work item and packs
 * the rows of several requests into one item, which pays where the shared
 * keys dominate.  The rule, set from measurements on MI355X: *use = 1 when
 * the batch is prefill-shaped (max_q_len * Hq/Hkv > 32 query columns per
 * request and kv head), shared_len covers at least three 64-key tiles and no
 * request has more than 128 keys past it (seq_lens[r] - shared_len <= 128);
 * else 0.  Decode-shaped batches keep the single pass.
 *
 * seq_lens   [host] int32 [B]  context length L_r of each request, >= shared_len
 * max_q_len, Hq, Hkv  as for ilpc_paged_prefill_attn
 * shared_len as ilpc_shared_prefix_len returned it
 * use        out: 1 or 0 (0 for B = 0)
 * ILPC_EINVAL for NULL pointers, B < 0, shared_len < 0, max_q_len < 0, head
 * counts that do not divide, or a request shorter than shared_len.
 */
int ilpc_prefer_shared_split(const int32_t* seq_lens, int32_t B, int32_t max_q_len, int32_t Hq, int32_t Hkv,
                             int32_t shared_len, int32_t* use);

/*
 * Prefix-aware refinement of in-context demonstrations (section 3.2.1, with
 * its matching / modifying / reordering figure, and section 3.2.2 on the ICL
 * table).  Host only,
 * synchronous; the table is library-owned host memory.
 *
 * A demonstration is a (template id, demonstration id) pair of int32 values:
 * the template it is labelled with and the concrete log (so, its tokens).  A
 * demonstration set (DS) is an ordered list of n_demos of them.  The ICL table
 * keeps the sets of past requests in least-recently-used order.
 */
typedef struct ilpc_pair_table ilpc_pair_table; /* opaque, host memory, library-owned */

/* Create an empty ICL table holding at most `capacity` sets (1 .. 2^24) of
 * `n_demos` demonstrations (1 .. 4096).  *out receives the handle (NULL on
 * error).  All of the table's memory is taken here: ILPC_ENOSPC if the host
 * cannot provide it, ILPC_EINVAL for sizes out of range. */
int ilpc_pair_create(int32_t capacity, int32_t n_demos, ilpc_pair_table** out);

/* Free a table (NULL is ignored). */
void ilpc_pair_destroy(ilpc_pair_table* table);

/* Empty the table. */
int ilpc_pair_reset(ilpc_pair_table* table);

/*
 * Refine B requests' demonstration sets in order, each against the table as
 * the previous requests left it (a request's set enters the table as after
 * its inference completed).
 *
 * templates, demos         [host] int32 [B*n_demos]  current sets, request-major
 * out_templates, out_demos [host] int32 [B*n_demos]  out: final sets
 * pmc                      [host] int32 [B]          out: prefix-matching count
 *
 * PMC of a past set H against the current set C: the number of leading
 * demonstrations of H whose templates all occur in C, each demonstration of
 * C serving at most one of them.  The target is the past set of largest PMC,
 * ties going to the most recently used; PMC 0 means no target.  Final set:
 * the target's first PMC demonstrations in the target's order (each replacing
 * the first not yet replaced current demonstration of its template), then
 * the remaining current demonstrations in their order.  Table update:
 * PMC = n_demos reuses the target (final = target) and makes it the most
 * recently used; PMC = 0 appends the current set unchanged; otherwise the
 * final set is appended and the target keeps its place.  A set already held
 * is stored once (appending it refreshes it); beyond the capacity the least
 * recently used set is evicted.  Errors (NULL table or pointer, negative B:
 * ILPC_EINVAL) are reported before anything changes; otherwise the call
 * completes, since every structure the table uses was sized by
 * ilpc_pair_create and refinement allocates nothing.
 */
int ilpc_pair_refine(ilpc_pair_table* table, const int32_t* templates, const int32_t* demos, int32_t B,
                     int32_t* out_templates, int32_t* out_demos, int32_t* pmc);

/* Copy the held sets, least recently used first, into templates / demos
 * [host] int32 [max_entries*n_demos]; *n_entries receives their number
 * (ILPC_EINVAL, with *n_entries set, if they do not fit). */
int ilpc_pair_entries(const ilpc_pair_table* table, int32_t* templates, int32_t* demos, int32_t max_entries,
                      int32_t* n_entries);

#ifdef __cplusplus
}
#endif

#endif /* ILPC_H */
