/*
 * ws_attn.h -- C ABI of the block-causal streaming attention library
 * (libwsattn.so, gfx950 / MI355X).
 *
 * The operation (Wan-Streamer v0.1, Abstract, Sec. 1 with Fig. 1, Sec. 5):
 * one Transformer runs over an interleaved stream of visual, audio and text
 * tokens grouped into streaming units ("blocks"); attention is block-causal:
 * every token sees all tokens of its own block (both directions) and every
 * token of every earlier block, and nothing later.  Sec. 2.1, Eq. 1 gives the
 * same conditioning set (unit k conditions on inputs of units <= k and on
 * responses of units < k).  Sec. 2.4: after the system prefill the
 * performer keeps a full-history KV cache, appends each received KV slice to
 * it, and runs the flow-matching solver for the next unit against it; the
 * current (noisy) unit is not yet part of the cache (Sec. 2.1: clean latents
 * are appended after denoising).
 *
 * For query i with block id beta(i) and keys j with block ids beta(j):
 *   o_i   = sum_{j : beta(j) <= beta(i)} softmax_j(scale * <q_i, k_j>) v_j
 *   lse_i = natural log of the softmax denominator (including its max shift)
 * Grouped-query attention: query head h reads KV head h / (Hq / Hkv).
 *
 * Token-causal segments (the *_text entry points).  The thinker decodes the
 * language and state slots of a unit token by token (Sec. 1, Sec. 2.4;
 * language is trained by next-token prediction, Sec. 2.1).  A block may end
 * in such a segment, starting at position tau of the block: the block's
 * tokens before tau (its observations) see each other in both directions
 * but not the segment, and a segment token at position i sees the
 * observations and the segment tokens at positions <= i.  Earlier blocks
 * stay fully visible.  So token i of a block sees exactly the keys
 * j < max(tau, i + 1); tau = block end means no segment (plain
 * block-causal), tau = block start makes the block token-causal.
 *
 * New blocks of different lengths (the *_varlen entry points).  Units hold
 * varying numbers of visual, audio and text tokens (Sec. 2.2), so
 * concurrent streams stepped in one launch carry new blocks of different
 * lengths, padded to a common new_len.  Padding tokens are never keys and
 * are never committed; the outputs of their rows are unspecified.
 *
 * Conventions for every entry point
 * ---------------------------------
 * - Token tensors are 4-d [batch][tokens][heads][head_dim] described by
 *   ws_tensor4: the head_dim axis is contiguous; the three other strides are
 *   in ELEMENTS.  Pointers must be 16-byte aligned and strides multiples of
 *   8 elements (128-bit loads).  The keys and values read by the attention
 *   entry points (k_new / v_new of a step, k / v of a prefill) must have a
 *   token stride below 2^24 elements (WS_ERR_SHAPE otherwise): the kernels
 *   address a tile of them with 32-bit offsets.
 * - All device pointers are HIP device memory of the current device; the
 *   caller owns every buffer (inputs, outputs, cache pool, page tables,
 *   workspace).  The library allocates no device memory and keeps no state
 *   between calls except its loaded code object (which holds the scratch
 *   array of ws_block_causal_attn_fwd_noalloc) and, per device, the
 *   compute-unit count and that array's address, looked up once.
 * - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *   All device work is enqueued on it; the call returns after enqueueing
 *   (stream-ordered, asynchronous).  Host arrays are read only during the
 *   call.  Calls that write the same memory must be ordered by the caller.
 * - Every argument is validated on the host before anything is enqueued.
 *   A non-zero return from validation guarantees that no byte of any
 *   output, lse, cache pool or workspace was changed.  WS_ERR_HIP reports a
 *   HIP launch error after validation passed.  Nothing is thrown or aborted
 *   across the ABI.  ws_last_error() gives a human-readable reason.
 * - Supported: head_dim 64 or 128; inputs bf16; outputs bf16 or f32;
 *   page_size 64.
 * - The attention and append entry points enqueue kernels only (no device
 *   allocation, no synchronisation, no memset), so a caller may record them
 *   into a HIP graph by stream capture, e.g. the performer's solver loop of a
 *   unit (Sec. 2.4).  A replay repeats the recorded call exactly: the host
 *   arrays (cache lengths, page ids, offsets, segment starts, new-block
 *   lengths) are read when the call is recorded, and small batches pass
 *   cache lengths, segment starts and new-block lengths to the kernels by
 *   value.
 * - A call with no token to process (batch == 0, or new_len / seq_len == 0)
 *   returns WS_OK after checking its scalar arguments, enqueues nothing and
 *   accepts NULL tensor pointers.
 */
#ifndef WS_ATTN_H
#define WS_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WS_ABI_VERSION 5
#define WS_PAGE_SIZE 64

typedef enum {
    WS_OK = 0,
    WS_ERR_NULL = 1,        /* a required pointer is NULL                    */
    WS_ERR_SHAPE = 2,       /* a size is negative or sizes are inconsistent  */
    WS_ERR_UNSUPPORTED = 3, /* head_dim, dtype or page_size not supported    */
    WS_ERR_ALIGN = 4,       /* pointer not 16-byte aligned / stride % 8 != 0 */
    WS_ERR_OFFSETS = 5,     /* block offsets: first != 0, decreasing, last != seq_len;
                               or a token-causal segment start outside its block */
    WS_ERR_PAGE = 6,        /* a page id that would be touched is outside [0, num_pages) */
    WS_ERR_CAPACITY = 7,    /* tokens exceed max_pages_per_seq * page_size   */
    WS_ERR_HEADS = 8,       /* num_q_heads % num_kv_heads != 0, or head counts differ from the cache's */
    WS_ERR_WORKSPACE = 9,   /* workspace NULL or smaller than ws_workspace_bytes() */
    WS_ERR_HIP = 10         /* the HIP runtime reported an error            */
} ws_status;

enum { WS_DTYPE_BF16 = 1, WS_DTYPE_F32 = 2 };

/* flags of ws_block_causal_attn_fwd */
enum { WS_FUSE_APPEND = 1 };

/* op codes of ws_workspace_bytes */
enum { WS_OP_STEP = 1, WS_OP_PREFILL = 2, WS_OP_PREFILL_BWD = 3 };

/* A [batch][tokens][heads][head_dim] tensor; head_dim contiguous; strides in elements. */
typedef struct {
    void *ptr;
    int32_t dtype; /* WS_DTYPE_BF16 or WS_DTYPE_F32 */
    int64_t stride_b, stride_t, stride_h;
} ws_tensor4;

/*
 * Paged full-history KV cache (Sec. 2.4: the performer's full-history
 * cache).  k_pool and v_pool are bf16 [num_pages][num_kv_heads][page_size]
 * [head_dim], contiguous: one (page, KV head) is page_size * head_dim
 * consecutive elements.  Logical token position p of stream b lives in
 * physical page page_table[b][p / page_size], slot p % page_size.
 * page_table_dev and page_table_host hold the same [batch][max_pages_per_seq]
 * int32 table (device copy read by kernels, host copy validated by the
 * library; the caller keeps them equal).  Entries are only read for
 * positions that a call touches.
 */
typedef struct {
    void *k_pool;
    void *v_pool;
    const int32_t *page_table_dev;
    const int32_t *page_table_host;
    int32_t num_pages;
    int32_t page_size;          /* must be WS_PAGE_SIZE */
    int32_t max_pages_per_seq;
    int32_t num_kv_heads;
    int32_t head_dim;
} ws_paged_kv;

/* WS_ABI_VERSION of the loaded library. */
int ws_abi_version(void);

/* Static name of a status code ("WS_OK", "WS_ERR_SHAPE", ...). */
const char *ws_status_string(int status);

/* Reason for the last non-OK status returned on this thread ("" if none). */
const char *ws_last_error(void);

/*
 * ws_kv_append -- commit one block of new tokens to the paged cache
 * (Sec. 2.4: the performer appends the received KV slice to its
 * full-history cache; Sec. 2.1: clean latents are appended to the history).
 *
 * For every stream b < batch and token t < new_len, copies k_new[b][t][h][:]
 * and v_new[b][t][h][:] (all KV heads h) bit for bit to logical position
 * cache_lens[b] + t of stream b.  k_new / v_new: bf16 [batch][new_len]
 * [num_kv_heads][head_dim].  cache_lens_host / cache_lens_dev: int32
 * [batch], the same values on host (validated) and device.  The cache
 * lengths are not updated; the caller adds new_len afterwards.
 * Errors: WS_ERR_NULL, WS_ERR_SHAPE (batch/new_len < 0, cache_lens < 0),
 * WS_ERR_UNSUPPORTED, WS_ERR_ALIGN, WS_ERR_CAPACITY, WS_ERR_PAGE, WS_ERR_HIP.
 */
int ws_kv_append(const ws_paged_kv *kv, int32_t batch,
                 const int32_t *cache_lens_host, const int32_t *cache_lens_dev,
                 int32_t new_len, ws_tensor4 k_new, ws_tensor4 v_new, void *stream);

/*
 * ws_block_causal_attn_fwd -- one streaming step (Sec. 2.4 and Fig. 2: the
 * performer's solver runs the current unit against the full-history cache;
 * Sec. 2.1: the current unit is noisy and attends to the clean context).
 *
 * The new_len tokens of the new block of stream b see the cache tokens
 * [0, cache_lens[b]) (all earlier blocks) and all new_len tokens of the new
 * block itself.  No key is masked except past the end.
 *   q:           bf16 [batch][new_len][num_q_heads][head_dim]
 *   k_new/v_new: bf16 [batch][new_len][num_kv_heads][head_dim]; the block's
 *                own keys and values, read from here (not from the cache)
 *   kv:          the paged cache; num_kv_heads and head_dim come from it
 *   cache_lens:  int32 [batch] on host and device, same values
 *   scale:       multiplies <q, k> (1/sqrt(head_dim) by convention)
 *   flags:       WS_FUSE_APPEND also commits k_new/v_new at cache_lens in the
 *                same launch (as ws_kv_append would); the attention result
 *                is identical.  cache_lens are not updated.
 *   out:         bf16 or f32 [batch][new_len][num_q_heads][head_dim]
 *   lse:         NULL or device f32 [batch][num_q_heads][new_len]
 *   workspace:   device scratch of at least
 *                ws_workspace_bytes(WS_OP_STEP, batch, num_q_heads,
 *                kv->num_kv_heads, new_len, max_b cache_lens[b] + new_len)
 *                bytes (NULL allowed when that is 0); its contents on entry
 *                are ignored.
 * new_len x (num_q_heads / num_kv_heads) must not exceed 2^30 (WS_ERR_SHAPE).
 * The library splits long caches into KV partitions merged by a second
 * launch.  The partition count is planned for the compute units of the
 * current device (queried once per device; ws_step_plan shows the plan for
 * any count).  The environment variable WS_SPLITS (1..32) overrides it for
 * tuning; it is read once per process, at the first call that plans a
 * step, so workspace queries and calls always agree.
 * Errors: WS_ERR_NULL, WS_ERR_SHAPE, WS_ERR_UNSUPPORTED, WS_ERR_ALIGN,
 * WS_ERR_HEADS, WS_ERR_CAPACITY, WS_ERR_PAGE, WS_ERR_WORKSPACE, WS_ERR_HIP.
 */
int ws_block_causal_attn_fwd(ws_tensor4 q, ws_tensor4 k_new, ws_tensor4 v_new,
                             const ws_paged_kv *kv,
                             const int32_t *cache_lens_host, const int32_t *cache_lens_dev,
                             int32_t batch, int32_t new_len, int32_t num_q_heads,
                             float scale, int32_t flags,
                             ws_tensor4 out, float *lse,
                             void *workspace, size_t workspace_bytes, void *stream);

/*
 * ws_block_causal_attn_fwd_noalloc -- ws_block_causal_attn_fwd for callers
 * that cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation.  It allocates nothing
 * (no hipMalloc, hipFree or allocating library call): the split-KV partials
 * go to a scratch array of WS_NOALLOC_SCRATCH_BYTES that the library's code
 * object holds on each device (until the process ends) instead of a caller
 * workspace.  Same arguments, results and errors as ws_block_causal_attn_fwd
 * without workspace / workspace_bytes; a step whose plan needs more partial
 * storage than the array holds (ws_step_plan reports it) gives
 * WS_ERR_WORKSPACE.  Every call on a device shares that device's array and
 * nothing in it needs to start at zero (each call writes the partials it
 * reads); calls that may overlap on one device (unordered streams) race on
 * it and give undefined results, so order them.
 */
#define WS_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int ws_block_causal_attn_fwd_noalloc(ws_tensor4 q, ws_tensor4 k_new, ws_tensor4 v_new,
                                     const ws_paged_kv *kv,
                                     const int32_t *cache_lens_host, const int32_t *cache_lens_dev,
                                     int32_t batch, int32_t new_len, int32_t num_q_heads,
                                     float scale, int32_t flags,
                                     ws_tensor4 out, float *lse, void *stream);

/*
 * ws_block_causal_prefill -- block-causal attention over whole sequences
 * (Sec. 2.4: the system prefill that builds the initial full-history state;
 * Sec. 2.3: training uses the same causal format as inference).
 *
 * Every stream holds seq_len tokens split into num_blocks consecutive blocks
 * with boundaries block_offsets[b][0..num_blocks] (first 0, non-decreasing,
 * last seq_len; zero-length blocks are allowed and own no token).  Token i
 * sees every token j < end of i's block.
 *   q:    bf16 [batch][seq_len][num_q_heads][head_dim]
 *   k, v: bf16 [batch][seq_len][num_kv_heads][head_dim], or k.ptr == v.ptr ==
 *         NULL to read keys and values from kv_or_null (positions
 *         [0, seq_len) of each stream, e.g. filled by ws_kv_append)
 *   block_offsets_host / _dev: int32 [batch][num_blocks + 1], same values
 *   out:  bf16 or f32 [batch][seq_len][num_q_heads][head_dim]
 *   lse:  NULL or device f32 [batch][num_q_heads][seq_len]
 * Errors: WS_ERR_NULL, WS_ERR_SHAPE, WS_ERR_UNSUPPORTED, WS_ERR_ALIGN,
 * WS_ERR_HEADS, WS_ERR_OFFSETS, WS_ERR_CAPACITY, WS_ERR_PAGE, WS_ERR_HIP.
 */
int ws_block_causal_prefill(ws_tensor4 q, ws_tensor4 k, ws_tensor4 v,
                            const ws_paged_kv *kv_or_null,
                            const int32_t *block_offsets_host, const int32_t *block_offsets_dev,
                            int32_t batch, int32_t seq_len, int32_t num_blocks,
                            int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                            float scale, ws_tensor4 out, float *lse, void *stream);

/*
 * ws_block_causal_attn_fwd_text -- a streaming step whose new block ends in
 * a token-causal segment (the thinker's pass over the language and state
 * slots, Sec. 1 and Sec. 2.4).  Same arguments and errors as
 * ws_block_causal_attn_fwd, plus
 *   text_starts_host / _dev: int32 [batch], same values on host and device:
 *                the segment of stream b's new block starts at token
 *                text_starts[b] of the block, 0 <= text_starts[b] <= new_len
 *                (new_len: no segment; 0: the block is token-causal).  New
 *                token t sees cache tokens [0, cache_lens[b]) and new tokens
 *                [0, max(text_starts[b], t + 1)).
 * A start outside [0, new_len] gives WS_ERR_OFFSETS.  Workspace as for
 * ws_block_causal_attn_fwd.
 */
int ws_block_causal_attn_fwd_text(ws_tensor4 q, ws_tensor4 k_new, ws_tensor4 v_new,
                                  const ws_paged_kv *kv,
                                  const int32_t *cache_lens_host, const int32_t *cache_lens_dev,
                                  const int32_t *text_starts_host, const int32_t *text_starts_dev,
                                  int32_t batch, int32_t new_len, int32_t num_q_heads,
                                  float scale, int32_t flags,
                                  ws_tensor4 out, float *lse,
                                  void *workspace, size_t workspace_bytes, void *stream);

/*
 * ws_block_causal_attn_fwd_varlen -- a streaming step over streams whose new
 * blocks differ in length (concurrent streams, each at its own unit: blocks
 * hold varying numbers of visual, audio and text tokens, Sec. 2.2 and
 * Sec. 2.4), padded to a common new_len.  Same arguments and errors as
 * ws_block_causal_attn_fwd_text, plus
 *   new_lens_host / _dev: int32 [batch], same values on host and device:
 *                stream b's new block is its first new_lens[b] tokens,
 *                1 <= new_lens[b] <= new_len; tokens past it are padding.
 *   text_starts_host / _dev: as for ws_block_causal_attn_fwd_text, or both
 *                NULL for no segment.
 * New token t of stream b sees cache tokens [0, cache_lens[b]) and new tokens
 * [0, min(new_lens[b], max(text_starts[b], t + 1))): padding is never a key
 * (never read, so its contents do not matter) and, with WS_FUSE_APPEND, never
 * committed: only positions [cache_lens[b], cache_lens[b] + new_lens[b]) of
 * the cache are written.  The outputs and lse of padding rows are
 * unspecified: query tiles holding padding only are skipped (no work, no
 * store), so a short block costs about its own length, not new_len.
 * A length outside [1, new_len] gives WS_ERR_SHAPE.  workspace: at least
 * ws_step_workspace_bytes_varlen(batch, num_q_heads, kv->num_kv_heads,
 * new_len, cache_lens_host, new_lens_host) bytes (the KV split count
 * depends on the lengths, so ws_workspace_bytes does not give it).
 */
int ws_block_causal_attn_fwd_varlen(ws_tensor4 q, ws_tensor4 k_new, ws_tensor4 v_new,
                                    const ws_paged_kv *kv,
                                    const int32_t *cache_lens_host, const int32_t *cache_lens_dev,
                                    const int32_t *new_lens_host, const int32_t *new_lens_dev,
                                    const int32_t *text_starts_host, const int32_t *text_starts_dev,
                                    int32_t batch, int32_t new_len, int32_t num_q_heads,
                                    float scale, int32_t flags,
                                    ws_tensor4 out, float *lse,
                                    void *workspace, size_t workspace_bytes, void *stream);

/*
 * ws_step_workspace_bytes_varlen -- device workspace bytes that
 * ws_block_causal_attn_fwd_varlen needs for these host arrays (int32
 * [batch] each), planned for the current device.  0 when none is needed,
 * when an argument is invalid (the call itself then reports why) or when
 * no device is available.
 */
size_t ws_step_workspace_bytes_varlen(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                      int32_t new_len, const int32_t *cache_lens_host,
                                      const int32_t *new_lens_host);

/*
 * ws_kv_append_varlen -- ws_kv_append for blocks of different lengths: only
 * tokens t < new_lens[b] of stream b are committed (new_lens_host / _dev:
 * int32 [batch], same values, 0 <= new_lens[b] <= new_len).  Same arguments
 * and errors as ws_kv_append; a length outside [0, new_len] gives
 * WS_ERR_SHAPE.
 */
int ws_kv_append_varlen(const ws_paged_kv *kv, int32_t batch,
                        const int32_t *cache_lens_host, const int32_t *cache_lens_dev,
                        const int32_t *new_lens_host, const int32_t *new_lens_dev,
                        int32_t new_len, ws_tensor4 k_new, ws_tensor4 v_new, void *stream);

/*
 * ws_block_causal_prefill_text -- whole sequences whose blocks end in
 * token-causal segments (the thinker's language and state slots, Sec. 1 and
 * Sec. 2.4).  Same arguments and errors as ws_block_causal_prefill, plus
 *   text_starts_host / _dev: int32 [batch][num_blocks], same values: the
 *          segment of block n of stream b starts at absolute token
 *          text_starts[b][n], block_offsets[b][n] <= text_starts[b][n] <=
 *          block_offsets[b][n+1] (the block end: no segment).  Token i of
 *          block n sees every token j < max(text_starts[b][n], i + 1).
 * A start outside its block gives WS_ERR_OFFSETS.
 */
int ws_block_causal_prefill_text(ws_tensor4 q, ws_tensor4 k, ws_tensor4 v,
                                 const ws_paged_kv *kv_or_null,
                                 const int32_t *block_offsets_host, const int32_t *block_offsets_dev,
                                 const int32_t *text_starts_host, const int32_t *text_starts_dev,
                                 int32_t batch, int32_t seq_len, int32_t num_blocks,
                                 int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                 float scale, ws_tensor4 out, float *lse, void *stream);

/*
 * ws_block_causal_prefill_bwd -- gradients of ws_block_causal_prefill(_text)
 * for training (Sec. 2.3: training uses the same causal format as
 * inference).  For an upstream gradient dO of the output, with P the
 * softmax weights of the forward (0 for masked keys):
 *   D_i = <dO_i, O_i>,  dS_ij = P_ij (<dO_i, v_j> - D_i),
 *   dQ_i = scale sum_j dS_ij k_j,  dK_j = scale sum_i dS_ij q_i,
 *   dV_j = sum_i P_ij dO_i,
 * the sums over i running over every query row and query head that reads
 * KV head floor(h / G).
 *   q, o, dout: bf16 [batch][seq_len][num_q_heads][head_dim]; o is the
 *               forward's output (its bf16 values enter D)
 *   k, v:       bf16 [batch][seq_len][num_kv_heads][head_dim] (contiguous
 *               keys; no paged variant)
 *   lse:        device f32 [batch][num_q_heads][seq_len], the forward's lse
 *   block_offsets_host / _dev: as ws_block_causal_prefill
 *   text_starts_host / _dev:   NULL / NULL for block-causal, or as
 *               ws_block_causal_prefill_text
 *   dq:         f32 [batch][seq_len][num_q_heads][head_dim] (written)
 *   dk, dv:     f32 [batch][seq_len][num_kv_heads][head_dim] (written)
 *   workspace:  device scratch of ws_workspace_bytes(WS_OP_PREFILL_BWD,
 *               batch, num_q_heads, num_kv_heads, seq_len, seq_len) bytes,
 *               16-byte aligned; contents on entry ignored
 * The gradients are deterministic (fixed summation order; no atomics).
 * Errors: WS_ERR_NULL, WS_ERR_SHAPE, WS_ERR_UNSUPPORTED, WS_ERR_ALIGN,
 * WS_ERR_HEADS, WS_ERR_OFFSETS, WS_ERR_WORKSPACE, WS_ERR_HIP.
 */
int ws_block_causal_prefill_bwd(ws_tensor4 q, ws_tensor4 k, ws_tensor4 v, ws_tensor4 o,
                                ws_tensor4 dout, const float *lse,
                                const int32_t *block_offsets_host, const int32_t *block_offsets_dev,
                                const int32_t *text_starts_host, const int32_t *text_starts_dev,
                                int32_t batch, int32_t seq_len, int32_t num_blocks,
                                int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                float scale, ws_tensor4 dq, ws_tensor4 dk, ws_tensor4 dv,
                                void *workspace, size_t workspace_bytes, void *stream);

/*
 * Workspace bytes ws_block_causal_attn_fwd (and its _text variant) needs
 * for this shape (op =
 * WS_OP_STEP; num_kv_heads = the cache's; max_k = largest cache_lens[b] +
 * new_len), planned for the current device's compute units (0 when no
 * device is available).  WS_OP_PREFILL returns 0.  WS_OP_PREFILL_BWD
 * (max_q = max_k = seq_len): the bytes ws_block_causal_prefill_bwd needs
 * (pure host arithmetic).  Returns 0 for invalid arguments.
 */
size_t ws_workspace_bytes(int32_t op, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                          int32_t max_q, int32_t max_k);

/*
 * ws_step_plan -- the launch plan of a streaming step (host only; nothing
 * is enqueued).  Work items are (stream, KV head, 256-row query tile, KV
 * split); the plan picks the KV split count for num_cus compute units
 * (0: the current device's) and reports the workspace the step needs:
 * the value ws_block_causal_attn_fwd(_text) (new_lens_host NULL) or
 * ws_block_causal_attn_fwd_varlen (new_lens_host: int32 [batch]) checks
 * on a device with that many compute units.
 *   cache_lens_host: int32 [batch]
 *   num_splits, workspace_bytes: outputs
 * Errors: WS_ERR_NULL, WS_ERR_SHAPE (sizes, a length outside its range),
 * WS_ERR_HEADS, WS_ERR_HIP (num_cus == 0 and no device).
 */
int ws_step_plan(int32_t num_cus, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                 int32_t new_len, const int32_t *cache_lens_host, const int32_t *new_lens_host,
                 int32_t *num_splits, size_t *workspace_bytes);

#ifdef __cplusplus
}
#endif

#endif /* WS_ATTN_H */
