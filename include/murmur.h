/*
 * libmurmur -- decode-step GQA attention over a sliding-window-evicted KV cache
 * (Murmur, "An Efficient Inference System for Long-Form ASR", Section 3.2).
 *
 * An LLM-based ASR decoder keeps, per sequence (one audio chunk), a KV cache
 * laid out as [system prompt][speech tokens][system prompt][output tokens]
 * (Section 3.2, the sequence structure paragraph).  At every decode step only a
 * positional subset of that cache is attended: the system prompts, a window of
 * speech tokens that starts to advance after a delay (Algorithm 2, with the
 * speech sinks of Equation 2), and StreamingLLM-style sinks plus a recent
 * window of output tokens (Algorithm 1).  The current token attends over the
 * kept entries with ordinary softmax attention (Equation 1).
 *
 * Two calls form the hot path of one decode step:
 *   murmur_evict_compact  -- policy -> per-sequence retained-position lists
 *                            (and an equivalent table of contiguous ranges);
 *   murmur_decode_attn    -- split-K grouped-query attention over those
 *                            positions with a log-sum-exp merge of the splits.
 * murmur_decode_step does both in one launch (murmur_decode_step_static too,
 * without a workspace argument); murmur_decode_step_ring does it
 * on physical eviction storage (an output ring) and appends the current
 * token's K/V; murmur_evict_compact_paged emits the lists as rows of a paged
 * pool.  Host-only helpers size the lists, lay out ring storage, name the
 * paged blocks no later step reads, and plan the chunking of a long recording
 * (Section 3.1, Equation 4).
 *
 * Conventions shared by every call:
 *   - Pointers named *_dev are device memory (HIP, the current device); all
 *     other pointers are host memory.  Every buffer is owned by the caller;
 *     the library keeps no pointer after a call returns and allocates nothing
 *     (murmur_decode_step_static uses a scratch array of the library's own,
 *     see there).
 *   - Hot calls are asynchronous on `stream` (NULL = the null stream), never
 *     synchronise the host, issue only kernel launches, and may be captured
 *     into a HIP graph.
 *   - Return value: MURMUR_OK (0) or a negative MURMUR_E* code.  All argument
 *     checks run before any HIP call, so a rejected call touches no device
 *     state.  murmur_last_error() then describes the failure.
 *   - Conditions only the device can see (a retained count above max_keep, a
 *     position outside the cache, an invalid per-sequence policy) set bits in
 *     a per-device error word read by murmur_device_error(); the affected
 *     sequence's outputs are written as NaN so the failure is never silent.
 */
#ifndef MURMUR_H
#define MURMUR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Same object as hipStream_t; declared here so the header needs no HIP headers. */
typedef struct ihipStream_t *murmur_stream_t;

enum {
    MURMUR_OK = 0,
    MURMUR_EINVAL = -1,       /* a pointer, size, stride or policy value is invalid */
    MURMUR_EUNSUPPORTED = -2, /* valid but not implemented (head_dim != 128, group > 16, dtype) */
    MURMUR_ENOSPACE = -3,     /* max_keep below a retained count, or workspace too small */
    MURMUR_EHIP = -4,         /* a HIP runtime call failed; the message has hipGetErrorString */
};

enum { MURMUR_DTYPE_BF16 = 1, MURMUR_DTYPE_F32 = 2 };

/* Policy array layouts (the pol_per_seq argument, a bit set).  The array holds
 * [per layer ? n_layers : 1][per sequence ? B : 1] murmur_policy records;
 * (layer, sequence b) uses record
 *   (PER_LAYER ? layer * (PER_SEQ ? B : 1) : 0) + (PER_SEQ ? b : 0).
 * PER_LAYER is accepted by the fused steps only (the paper finds the speech
 * sparsity on 24 of its model's 28 layers, Section 1 and Section 2.3, so a
 * model may keep some layers dense); it makes their retained-set outputs
 * per layer too. */
enum { MURMUR_POL_PER_SEQ = 1, MURMUR_POL_PER_LAYER = 2 };

/* Device error word bits (murmur_device_error). */
enum {
    MURMUR_DEVERR_OVERFLOW = 1,  /* evict_compact: retained count > max_keep */
    MURMUR_DEVERR_POLICY = 2,    /* evict_compact: invalid layout or policy for a sequence */
    MURMUR_DEVERR_POSITION = 4,  /* decode_attn: retained position outside [0, max_len) */
    MURMUR_DEVERR_COUNT = 8,     /* decode_attn: count outside [1, max_keep] */
    MURMUR_DEVERR_CAPACITY = 16, /* decode_step_ring: the output ring cannot hold the retained outputs */
    MURMUR_DEVERR_BLOCK = 32,    /* evict_compact_paged: a retained position past the block table or in a freed block */
    MURMUR_DEVERR_POOL = 64,     /* paged_step: the free stack ran out (or overflowed its capacity) */
};

/* One sequence (audio chunk) of the batch, Section 3.2's layout
 * [prompt_pre][speech_len speech tokens][prompt_mid][out_len output tokens].
 * out_len is the paper's decode-step index j (>= 1): it counts the token being
 * generated, whose K/V the caller has already appended at output slot j-1.
 * Global positions are 0-based: speech starts at prompt_pre, output at
 * prompt_pre + speech_len + prompt_mid. */
typedef struct murmur_seg {
    int32_t prompt_pre;
    int32_t speech_len;
    int32_t prompt_mid;
    int32_t out_len;
} murmur_seg;

/* Eviction policy of one sequence (Section 3.2).
 *   speech_window  w of Algorithm 2 (>= 1), or -1 to keep every speech token;
 *   speech_delay   d of Algorithm 2 (>= 0): the window starts at speech token
 *                  l_j = max(0, j - max(d,1) + 1), i.e. 0 while j < d and one
 *                  further per step from j = d on, clamped to speech_len - w so
 *                  the window ends no later than the last speech token;
 *   speech_sink    n_sink of Equation 2 (>= 0): the first speech tokens, always kept;
 *   out_window     w of Algorithm 1 (>= 1), or -1 to keep every output token;
 *   out_sink       n_sink of Algorithm 1 (>= 0), counted from the first output token.
 * Both system prompts are always kept.  The retained set is a pure function of
 * (murmur_seg, murmur_policy): no state is carried between steps. */
typedef struct murmur_policy {
    int32_t speech_window;
    int32_t speech_delay;
    int32_t speech_sink;
    int32_t out_window;
    int32_t out_sink;
} murmur_policy;

/* One layer-stacked KV cache (Section 3.2: K, V in R^{L x d} per layer).
 * Element (layer, b, kv_head, pos, e) of K lives at
 *   k + layer*stride_layer + b*stride_b + kv_head*stride_h + pos*stride_pos + e
 * (strides in bf16 elements; the head_dim stride is 1).  V uses the same
 * strides.  max_len bounds the positions that may be read: every retained
 * position must lie in [0, max_len).  Both base pointers must be 16-byte
 * aligned and stride_layer, stride_b, stride_h, stride_pos multiples of 8. */
typedef struct murmur_kv {
    const void *k;
    const void *v;
    int32_t n_layers;
    int32_t max_len;
    int64_t stride_layer;
    int64_t stride_b;
    int64_t stride_h;
    int64_t stride_pos;
} murmur_kv;

/* ABI version of this header (bumped on any signature change). */
#define MURMUR_ABI_VERSION 10
int murmur_abi_version(void);

/* Text of the last failure on the calling thread; valid until the next call
 * on that thread.  Empty string after a successful call. */
const char *murmur_last_error(void);

/* Host-only sizing (no GPU needed).  Computes the retained count of each of
 * the B sequences -- prompts + |speech sinks U speech window| + |output sinks
 * U output window| (Algorithms 1 and 2, Equation 2) -- into counts[B] and
 * their maximum into *max_count.
 *   seg: host [B]; pol: host [pol_per_seq ? B : 1]; counts: host [B] or NULL.
 * Errors: MURMUR_EINVAL for a negative length, out_len < 1, speech_window or
 * out_window outside {-1} U [1, inf), a negative delay or sink count, or
 * pol_per_seq not 0/1. */
int murmur_retained_count_host(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq,
                               int32_t B, int32_t *counts, int32_t *max_count);

/* Applies the eviction policy on the device (Algorithm 1, Algorithm 2,
 * Equation 2) and emits, per sequence b:
 *   idx_dev[b*max_keep + r], r < count: the r-th retained global position,
 *       ascending and without duplicates; slots r >= count hold -1;
 *   count_dev[b]: the retained count;
 *   ranges_dev (nullable) [b][6][2]: the same set as six (start, length)
 *       pieces in ascending position order -- prompt_pre, speech sinks, speech
 *       window, prompt_mid, output sinks, output window -- non-overlapping,
 *       lengths >= 0, summing to count.
 *   seg_dev: device [B]; pol_dev: device [pol_per_seq ? B : 1].
 * Host errors: MURMUR_EINVAL (null pointers, B < 1, max_keep < 1,
 * pol_per_seq not 0/1).  Device errors: MURMUR_DEVERR_POLICY (count 0 and all
 * slots -1 for that sequence), MURMUR_DEVERR_OVERFLOW (count holds the true
 * count, idx the first max_keep positions). */
int murmur_evict_compact(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq,
                         int32_t B, int32_t *idx_dev, int32_t max_keep, int32_t *count_dev,
                         int32_t *ranges_dev, murmur_stream_t stream);

/* Paged KV cache (the block tables of a paged-attention engine such as vLLM,
 * the paper's second engine, Section 3.1): every sequence's positions live
 * in blocks of block_size rows of one shared pool, position p of sequence b
 * in pool row block_table[b][p / block_size] * block_size + p % block_size.
 * murmur_evict_compact_paged emits the retained set of every sequence (as
 * murmur_evict_compact) with the index list in pool rows, ready for
 * murmur_decode_attn in index-list mode over a murmur_kv that describes the
 * pool as one sequence of rows: stride_b = 0, max_len = pool rows, and for a
 * pool laid out [block][slot][kv_head][D] stride_pos = Hkv*D, stride_h = D
 * (or [kv_head][block][slot][D]: stride_pos = D, stride_h = pool rows * D).
 *   block_table_dev: device int32 [B][max_blocks], physical block numbers;
 *   block_size: a power of two;
 *   count_dev, ranges_dev: as murmur_evict_compact (ranges in sequence
 *               positions, not pool rows).
 * Errors as murmur_evict_compact; device error MURMUR_DEVERR_BLOCK (entry -1)
 * for a retained position past max_blocks blocks, in a block whose table
 * entry is negative (a freed block, see murmur_freeable_blocks_host), or in a
 * pool row beyond 2^31 - 1.  Other table entries are not range-checked here:
 * a row outside the pool is reported by murmur_decode_attn
 * (MURMUR_DEVERR_POSITION, NaN outputs). */
int murmur_evict_compact_paged(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq,
                               int32_t B, const int32_t *block_table_dev, int32_t max_blocks, int32_t block_size,
                               int32_t *idx_dev, int32_t max_keep, int32_t *count_dev, int32_t *ranges_dev,
                               murmur_stream_t stream);

/* Host-only (no GPU): the logical blocks of each sequence that hold only
 * positions no decode step from out_len on retains again, so that a paged
 * cache can return them to its pool (Section 3.2: an evicted entry leaves the
 * KV cache).  These are the speech tokens behind the window that are not
 * speech sinks, and the output tokens older than the window that are not
 * output sinks: the window start of Algorithm 2 never decreases and the
 * window of Algorithm 1 only moves forward.  Speech ahead of the window stays,
 * since the window moves onto it.  blocks[b][2][2]: (first logical block,
 * number of blocks) of the speech part, then of the output part, where
 * logical block k holds positions [k*block_size, (k+1)*block_size); (0, 0)
 * when no whole block qualifies.  The result at
 * a later step contains the one at an earlier step, so a caller frees what is
 * new.  block_size >= 1; pol_per_seq 0 or 1 (as murmur_evict_compact).
 * Errors: MURMUR_EINVAL as murmur_retained_count_host. */
int murmur_freeable_blocks_host(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq, int32_t B,
                                int32_t block_size, int32_t *blocks);

/* One decode step of a paged cache's block manager, on the device, so that a
 * whole decode loop -- paging included -- can be captured into one HIP graph
 * (Section 3.2: evicted entries leave the KV cache).  For every sequence at
 * step out_len, in one launch:
 *   1. every block of block_table_dev that lies wholly inside the positions
 *      no step from out_len on retains (the ranges murmur_freeable_blocks_host
 *      names) and is still allocated (entry >= 0) is pushed onto the free
 *      stack, and its entry becomes -1;
 *   2. if the logical block of the current token (position
 *      prompt_pre + speech_len + prompt_mid + out_len - 1) has no block, one
 *      is popped for it (blocks freed in step 1 included);
 * and, with a pool, in a second launch:
 *   3. the current token's K and V are written into its pool row.
 * Call it once per decode step, in order, before murmur_evict_compact_paged;
 * every position before the current token must have a block (or have been
 * freed).  All pushes come before all pops, each in sequence order (placed by
 * block-wide scans), so the result is deterministic and a step's allocations
 * can use any block freed in that step.
 *   full_scan:       1: step 1 looks at every block of the ranges (the first
 *                    call after a prefill, or after steps were skipped);
 *                    0: only at the blocks that became whole since step
 *                    out_len - 1 (each later call: O(1) per sequence);
 *   block_table_dev: device int32 [B][max_blocks], physical block numbers,
 *                    -1 where there is none; updated in place;
 *   free_stack_dev:  device int32 [capacity], free physical blocks in
 *                    [0, *free_top_dev); capacity >= the pool's blocks;
 *   free_top_dev:    device int32, the number of free blocks; updated;
 *   pool:            nullable; the pool as murmur_decode_attn reads it in
 *                    index mode (stride_b ignored, max_len = pool rows);
 *   Hkv:             KV heads (with a pool);
 *   k_new_dev, v_new_dev: bf16 [n_layers][B][Hkv][128], contiguous, 16-byte
 *                    aligned (with a pool): the current token's K and V.
 * Errors: MURMUR_EINVAL (argument checks), MURMUR_EHIP.  Device errors:
 * MURMUR_DEVERR_POOL (the stack is empty: the entry stays -1, and so the
 * attention reports the position), MURMUR_DEVERR_BLOCK (the current token
 * lies past max_blocks), MURMUR_DEVERR_POLICY (that sequence is left as is). */
int murmur_paged_step(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq, int32_t B,
                      int32_t *block_table_dev, int32_t max_blocks, int32_t block_size, int32_t *free_stack_dev,
                      int32_t *free_top_dev, int32_t capacity, int32_t full_scan, const murmur_kv *pool,
                      int32_t Hkv, const void *k_new_dev, const void *v_new_dev, murmur_stream_t stream);

/* Workspace bytes murmur_decode_attn needs for these sizes and split_len
 * (0 = the automatic choice, or positions per split).
 * The workspace holds ticket counters (one per (layer, sequence, kv-head)
 * group that is split, and one per set of 8 splits of a group when the
 * LDS-staged schedule merges its 17 to 128 splits in two levels) in a region
 * at its start
 * whose size depends on ws_bytes alone (128 bytes per KiB, rounded up to 256),
 * and the split partials after that region.  It must be zero-filled once
 * before its first use (or reset with murmur_decode_attn_workspace_init);
 * every completed call leaves the tickets at zero again.  Calls of any shapes
 * may share a workspace as long as they pass the same ws_bytes (at least what
 * this function returns for each of them) and do not run concurrently. */
int murmur_decode_attn_workspace(int32_t n_layers, int32_t B, int32_t Hq, int32_t Hkv, int32_t max_keep,
                                 int32_t split_len, size_t *bytes);

/* Zeroes the ticket counters of a workspace with a small kernel (no memset
 * node, so it may be captured). */
int murmur_decode_attn_workspace_init(void *ws_dev, size_t ws_bytes, murmur_stream_t stream);

/* Decode-step attention (Equation 1) of the current token of every sequence,
 * in every layer, over the retained positions only:
 *   out[l,b,h,:] = sum_{i in R_b} softmax_i(scale * q[l,b,h,:] . K[l,b,g,i,:]) V[l,b,g,i,:]
 *   lse[l,b,h]   = log sum_{i in R_b} exp(scale * q[l,b,h,:] . K[l,b,g,i,:])
 * with g = h / (Hq/Hkv) (grouped-query attention, contiguous head groups) and
 * R_b the retained set of sequence b, shared by all layers and heads.
 *   q_dev:      bf16 [n_layers][B][Hq][D], contiguous, 16-byte aligned;
 *   kv:         host struct describing the bf16 K/V caches (see murmur_kv);
 *   ranges_dev: nullable [B][6][2] range table from murmur_evict_compact; when
 *               given it is used, each sequence's count is the table's total
 *               length (what murmur_evict_compact writes to count_dev), and
 *               neither idx_dev nor count_dev is read;
 *   idx_dev:    [B][max_keep] positions (used when ranges_dev is NULL);
 *   count_dev:  [B] retained counts (required with idx_dev; may be NULL with
 *               ranges_dev);
 *   D:          head_dim, must be 128; Hq/Hkv must be in [1, 16];
 *   scale:      logit scale (1/sqrt(D) for unscaled queries), finite;
 *   split_len:  the work schedule.  A positive multiple of 32: each (layer,
 *               sequence, KV head) is cut into splits of that many retained
 *               positions, one workgroup each (its four wavefronts take
 *               passes of 32 positions in turn), merged by log-sum-exp.
 *               0: automatic split length (at most one dispatch round of
 *               workgroups when the work is small, at most 64 splits per
 *               group otherwise);
 *   out_dev:    [n_layers][B][Hq][D] of out_dtype, 16-byte aligned
 *               (MURMUR_DTYPE_BF16 rounds to nearest even, MURMUR_DTYPE_F32
 *               stores the fp32 accumulation);
 *   lse_dev:    nullable fp32 [n_layers][B][Hq], natural log;
 *   ws_dev:     workspace of ws_bytes >= murmur_decode_attn_workspace(...).
 * Accumulation is fp32 throughout.  Errors: MURMUR_EINVAL, MURMUR_EUNSUPPORTED
 * (head_dim, group size, max_keep above 2^28), MURMUR_ENOSPACE (workspace),
 * MURMUR_EHIP; device errors
 * MURMUR_DEVERR_POSITION and MURMUR_DEVERR_COUNT. */
int murmur_decode_attn(const void *q_dev, const murmur_kv *kv, const int32_t *idx_dev, const int32_t *ranges_dev,
                       const int32_t *count_dev, int32_t max_keep, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                       float scale, int32_t split_len, void *out_dev, int32_t out_dtype, float *lse_dev,
                       void *ws_dev, size_t ws_bytes, murmur_stream_t stream);

/* One whole decode step in one launch: the retained set of every sequence
 * (Section 3.2: Algorithms 1-2 and Equation 2, as murmur_evict_compact) and
 * the attention over it (Equation 1, as murmur_decode_attn).  Each attention
 * workgroup derives its sequence's six pieces from seg_dev/pol_dev in closed
 * form, so nothing waits for a separate eviction launch; the results are
 * those of murmur_evict_compact followed by murmur_decode_attn with the range
 * table, bit for bit in the retained sets.
 *   seg_dev:    device [B], as murmur_evict_compact;
 *   pol_dev, pol_per_seq: device policy records in the layout the
 *               MURMUR_POL_* bits of pol_per_seq give (0..3);
 *   idx_dev, count_dev, ranges_dev: nullable outputs, written as
 *               murmur_evict_compact writes them (idx_dev [B][max_keep]),
 *               with MURMUR_POL_PER_LAYER one set per layer
 *               ([n_layers][B][max_keep], [n_layers][B], [n_layers][B][6][2]);
 *   split_len:  as murmur_decode_attn;
 *   every other argument: as murmur_decode_attn (same workspace size).
 * Device errors: MURMUR_DEVERR_POLICY and MURMUR_DEVERR_OVERFLOW as
 * murmur_evict_compact, MURMUR_DEVERR_COUNT for the same sequences (their
 * outputs are NaN), MURMUR_DEVERR_POSITION as murmur_decode_attn. */
int murmur_decode_step(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq,
                       const void *q_dev, const murmur_kv *kv, int32_t *idx_dev, int32_t *count_dev,
                       int32_t *ranges_dev, int32_t max_keep, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                       float scale, int32_t split_len, void *out_dev, int32_t out_dtype, float *lse_dev,
                       void *ws_dev, size_t ws_bytes, murmur_stream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * one-launch decode step of murmur_decode_step without a workspace argument.
 * Its tickets and split partials live in a scratch array of
 * MURMUR_STATIC_SCRATCH_BYTES that the library holds in device memory, one
 * copy per device, from the first call on that device until the process
 * ends; the call itself allocates and frees nothing.  On the first call on a
 * device the scratch's tickets are zeroed by a small kernel on `stream`;
 * every completed call leaves them at zero.  All calls on one device share
 * that device's scratch: calls that overlap in time on one device (other
 * streams, concurrent host threads) race and must not be issued.
 * Arguments, outputs and device errors: as murmur_decode_step.  Errors as
 * murmur_decode_step, plus MURMUR_ENOSPACE when the call's tickets and
 * partials (murmur_decode_attn_workspace for the same sizes and split_len)
 * exceed MURMUR_STATIC_SCRATCH_BYTES, and MURMUR_EHIP when the scratch's
 * address cannot be looked up. */
#define MURMUR_STATIC_SCRATCH_BYTES (4u << 20)
int murmur_decode_step_static(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq,
                              const void *q_dev, const murmur_kv *kv, int32_t *idx_dev, int32_t *count_dev,
                              int32_t *ranges_dev, int32_t max_keep, int32_t B, int32_t Hq, int32_t Hkv, int32_t D,
                              float scale, int32_t split_len, void *out_dev, int32_t out_dtype, float *lse_dev,
                              murmur_stream_t stream);

/* Physical eviction storage (Section 3.2: evicted entries leave the cache).
 * The output region of each sequence's cache holds its out_sink output sinks
 * at rows o0 .. o0+out_sink-1 (o0 = prompt_pre + speech_len + prompt_mid),
 * then a ring of out_capacity rows: 0-based output token i >= out_sink lives
 * at row o0 + out_sink + (i - out_sink) mod out_capacity.  A row is reused
 * only by a token that enters Algorithm 1's window after the row's previous
 * token has left it, so a cache of prompt_pre + speech_len + prompt_mid +
 * out_sink + out_capacity rows per sequence (instead of one row per generated
 * token) serves the whole decode.  Requirements per sequence: out_capacity
 * >= out_window when output eviction is on; with it off (out_window = -1),
 * out_len - out_sink <= out_capacity.  Prompt and speech rows are unchanged.
 *   out_capacity: ring rows (>= 1), the same for every sequence;
 *   k_new, v_new: device bf16 [n_layers][B][Hkv][D], contiguous, 16-byte
 *                 aligned: the current token's keys and values (the token
 *                 whose output index is out_len - 1). */
typedef struct murmur_ring {
    int32_t out_capacity;
    const void *k_new;
    const void *v_new;
} murmur_ring;

/* Host-only (no GPU): where the retained set of each sequence lies in ring
 * storage.  ranges[b][6][2] (nullable): six (start, length) row pieces that
 * hold exactly the tokens of murmur_evict_compact's pieces (same count):
 * prompt_pre, speech sinks, speech window, prompt_mid, then the output part
 * in at most two pieces -- piece 4 holds the output sinks and, when the
 * window wraps around the ring, its newer part (ring rows from 0), piece 5
 * the rest of the window.  cur_row[b] (nullable): the row of the current
 * token.  Errors: MURMUR_EINVAL as murmur_retained_count_host, or when the
 * ring cannot hold the retained outputs (see murmur_ring). */
int murmur_ring_layout_host(const murmur_seg *seg, const murmur_policy *pol, int32_t pol_per_seq, int32_t B,
                            int32_t out_capacity, int32_t *ranges, int32_t *cur_row);

/* One decode step on ring storage, in one launch: the retained set in
 * storage rows (as murmur_ring_layout_host), the attention of the current
 * token over it (Equation 1, as murmur_decode_step) and the append of the
 * current token's K/V into its ring row.  The attention reads the current
 * token from k_new/v_new, and no retained row is the one being written (it
 * held a token that has just left the window), so the append and the
 * attention do not race.  kv describes the ring storage (max_len >= the
 * rows above); the call writes row cur_row of every (layer, sequence, KV
 * head) of kv->k and kv->v, which must therefore be writable.
 *   idx_dev, count_dev, ranges_dev: nullable outputs as murmur_decode_step,
 *               in storage rows (idx in piece order, not ascending);
 *   pol_per_seq: MURMUR_POL_* bits as murmur_decode_step (the ring must hold
 *               the retained outputs of every layer's policy);
 *   split_len:  as murmur_decode_attn;
 *   every other argument: as murmur_decode_step.
 * Device errors: those of murmur_decode_step, and MURMUR_DEVERR_CAPACITY for
 * a sequence whose ring cannot hold its retained outputs (count 0, NaN
 * outputs, nothing appended). */
int murmur_decode_step_ring(const murmur_seg *seg_dev, const murmur_policy *pol_dev, int32_t pol_per_seq,
                            const murmur_ring *ring, const void *q_dev, const murmur_kv *kv, int32_t *idx_dev,
                            int32_t *count_dev, int32_t *ranges_dev, int32_t max_keep, int32_t B, int32_t Hq,
                            int32_t Hkv, int32_t D, float scale, int32_t split_len, void *out_dev,
                            int32_t out_dtype, float *lse_dev, void *ws_dev, size_t ws_bytes,
                            murmur_stream_t stream);

/* Chunked inference, host only (Section 3.1).  Packs the speech segments a
 * voice-activity detector found into chunks of at most max_chunk seconds,
 * greedily in time order, so that the chunks tile the recording from 0:
 * chunk i covers [chunk_start[i], chunk_start[i] + chunk_len[i]) and
 * chunk_start[i] is the sum of the lengths before it, the offset of
 * Equation 4.  A chunk takes the next segment while that segment ends within
 * max_chunk of the chunk's start; it then ends where the next segment begins
 * (so it keeps the silence after its last segment), or max_chunk after its
 * start if that comes first.  A segment longer than max_chunk is cut at
 * chunk boundaries; no other segment is cut (a chunk whose limit falls
 * inside such a segment ends where the segment begins, even if it then holds
 * only silence: the offsets need the tiling).  The last chunk ends at audio_len or max_chunk after its start,
 * whichever comes first; a recording without segments gives no chunk.
 *   seg_start, seg_end: [n_seg] seconds, 0 <= start < end <= audio_len,
 *               sorted by start, not overlapping (n_seg may be 0);
 *   chunk_start[i] equals the sum of chunk_len[0 .. i-1] up to rounding;
 *   chunk_of_seg: [n_seg] (nullable) chunk holding each segment's start;
 *   chunk_start, chunk_len: [max_chunks] outputs; *n_chunks: chunks written.
 *   speech_tokens (nullable): [max_chunks] speech tokens of each chunk at
 *               tokens_per_s (the speech_len of its murmur_seg: the chunk's
 *               length times the rate, rounded to nearest).
 * Errors: MURMUR_EINVAL (unsorted or overlapping segments, a segment outside
 * [0, audio_len], max_chunk <= 0, tokens_per_s < 0, audio_len / max_chunk or
 * n_seg above 2^24, max_chunk * tokens_per_s above 2e9), MURMUR_ENOSPACE (more
 * than max_chunks chunks; *n_chunks then holds the number needed). */
int murmur_plan_chunks(const double *seg_start, const double *seg_end, int32_t n_seg, double audio_len,
                       double max_chunk, double tokens_per_s, int32_t *chunk_of_seg, double *chunk_start,
                       double *chunk_len, int32_t *speech_tokens, int32_t max_chunks, int32_t *n_chunks);

/* Equation 4: absolute timestamps from chunk-relative ones,
 * t[k] = t_local[k] + offset(chunk[k]), offset(i) = chunk_len[0] + ... +
 * chunk_len[i-1].  Host only.  Errors: MURMUR_EINVAL for a chunk index
 * outside [0, n_chunks) or a negative chunk length. */
int murmur_chunk_timestamps(const double *t_local, const int32_t *chunk, int32_t n, const double *chunk_len,
                            int32_t n_chunks, double *t);

/* Measurement only (not part of the method): a plain read-only streaming
 * kernel, the practical ceiling the attention's achieved HBM bandwidth is
 * compared with.  n_workgroups workgroups of `threads` threads each read a
 * contiguous share of buf_dev[0, bytes) with 16-byte loads and keep an XOR of
 * what they read; sink_dev [n_workgroups] (4-byte aligned) is written only
 * if that XOR equals a fixed pattern, so the loads are not optimised away and
 * nearly nothing is written.  mode MURMUR_PROBE_REGISTERS: each thread issues
 * `depth` loads into registers, then waits for them; MURMUR_PROBE_LDS: the
 * loads go straight to LDS (the load type of the attention kernels), `depth`
 * per thread in flight at any time, using (threads / 64) * depth KiB of LDS.
 * buf_dev 16-byte aligned, bytes a positive multiple of 16, n_workgroups in
 * [1, 65535], threads a multiple of 64 in [64, 1024], depth 1, 2, 4, 8 or 16,
 * at most 64 KiB of LDS.  Errors: MURMUR_EINVAL, MURMUR_EHIP. */
#define MURMUR_PROBE_REGISTERS 0
#define MURMUR_PROBE_LDS 1
int murmur_read_probe(const void *buf_dev, size_t bytes, int32_t n_workgroups, int32_t threads, int32_t depth,
                      int32_t mode, uint32_t *sink_dev, murmur_stream_t stream);

/* Synchronises `stream`, returns the device error word of the current device
 * in *code (0 = none) and clears it.  Not for use inside a captured graph. */
int murmur_device_error(murmur_stream_t stream, int32_t *code);

#ifdef __cplusplus
}
#endif

#endif /* MURMUR_H */
