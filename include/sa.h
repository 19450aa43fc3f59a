/*
 * sa.h — C ABI of the segment re-prefill library (MI355X / gfx950).
 *
 * The library implements the data-parallel work behind lookahead context
 * engineering (SmoothAgent, arXiv 2607.00151): a context transformation
 * invalidates the KV cache and forces a re-prefill (paper Sec. 1, Sec. 3.1);
 * the lookahead stream builds the transformed segment's KV on top of the
 * already transformed prefix, in order (Sec. 3.2); at commit the transformed
 * prefix is spliced in place of the old one (Sec. 3.2, Listing of the agent
 * loop); keep-recent-K keeps the head of the context and its recent turns and
 * drops the run in between (Sec. 3.4).  The three data operations are:
 *
 *   sa_kv_assemble           commit splice: gather the surviving pages of a
 *                            cached context into fresh slots, in order, and
 *                            reserve room for the segment that follows
 *   sa_kv_append             write a new segment's K/V rows into the cache
 *   sa_segment_prefill_attn  causal grouped-query attention of the segment's
 *                            queries over the cached prefix plus, causally,
 *                            the segment itself (Sec. 4, prefill-attention
 *                            term: segment token i sees prefix + i + 1 keys)
 * and, fused from them, sa_kv_assemble_append (splice + append, one launch),
 * sa_segment_prefill_attn_append (append + attention, one launch) and the
 * copy-free splice sa_kv_splice_alias.
 *
 * Data layout (all device memory is owned by the caller):
 *   bf16 values are IEEE bfloat16 bit patterns (uint16).
 *   K pool, V pool  bf16 [num_layers][num_slots][num_kv_heads][page_size][head_dim]
 *                   (one slot holds page_size consecutive tokens of every KV head
 *                   of one layer; a slot id is the same in every layer)
 *   page table      CSR over sequences: the pages of sequence b are
 *                   indices[indptr[b] .. indptr[b+1]-1], logical token x of b is
 *                   row x % page_size of slot indices[indptr[b] + x / page_size]
 *   Q, O            bf16 [sum q_len][num_q_heads][head_dim], sequences back to back
 *   new K, V rows   bf16 [sum new_len][num_kv_heads][head_dim]
 *   LSE             fp32 [sum q_len][num_q_heads], natural log of the softmax
 *                   denominator of the scaled scores
 * Query head h reads KV head h / (num_q_heads / num_kv_heads).
 *
 * Conventions:
 *   - Lengths, spans and counts are small HOST int32 arrays, so grids are
 *     sized without a device round trip; page tables and free lists live on
 *     the device.
 *   - Every call validates its arguments on the host before touching HIP and
 *     returns a status; nothing throws across the ABI.  Validation order:
 *     layout and shapes, then pointers, then the context.
 *   - Calls enqueue work on `stream` (a hipStream_t; NULL is the default
 *     stream) and return without synchronising.  Buffers must stay valid until
 *     the stream has run the work.
 *   - A context keeps per-call plans (work lists) in device memory and reuses
 *     an uploaded plan when the next call of the same kind needs the same one.
 *     Calls on one context must therefore be ordered: use one stream per
 *     context (or one context per stream / thread).
 *   - Page ids inside device tables are range-checked by the kernels: a page
 *     beyond a sequence's list or a slot outside [0, num_slots) is skipped
 *     (never dereferenced) and latched in a device flag that sa_sync_check
 *     reports.  Reads of such pages contribute zeros.  Nothing on the hot
 *     path checks that slots do not repeat; with the environment variable
 *     SA_DEBUG=1 (read once per process) every splice and append first copies
 *     the tables it will use back to the host (synchronising its stream) and
 *     refuses, before launching, slots outside the pool or pages a sequence
 *     lacks (SA_ERR_RANGE), a free list that repeats a slot or hands out a
 *     surviving source slot, and two sequences writing the same row of a slot
 *     (SA_ERR_OVERLAP).
 *   - Plan buffers grow on demand (hipMalloc) and an outgrown one is kept
 *     until sa_destroy, since kernels already enqueued may still read it; no
 *     call synchronises the device.  sa_reserve sizes them ahead of time.
 *   - Pointers to pools, Q, O, K/V rows must be 16-byte aligned.
 */
#ifndef SA_H
#define SA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum sa_status {
    SA_OK = 0,
    SA_ERR_NULL = 1,          /* a required pointer (or the context) is NULL            */
    SA_ERR_SHAPE = 2,         /* inconsistent sizes or lengths                          */
    SA_ERR_UNSUPPORTED = 3,   /* head_dim != 128, page_size not 16 or 32, ...          */
    SA_ERR_ALIGN = 4,         /* a data pointer is not 16-byte aligned                  */
    SA_ERR_RANGE = 5,         /* a span or page id is out of range                      */
    SA_ERR_NO_PAGES = 6,      /* free list or destination table too small               */
    SA_ERR_HIP = 7,           /* a HIP runtime call failed (see sa_last_error)          */
    SA_ERR_DEVICE = 8,        /* no usable gfx950 device                                 */
    SA_ERR_OVERLAP = 9        /* slot lists repeat where they must not (SA_DEBUG checks) */
} sa_status;

typedef struct sa_ctx sa_ctx;

/* Cache geometry shared by every call that touches the pools. */
typedef struct sa_layout {
    int32_t num_q_heads;      /* Hq, a multiple of num_kv_heads                         */
    int32_t num_kv_heads;     /* Hkv >= 1                                               */
    int32_t head_dim;         /* must be 128                                            */
    int32_t page_size;        /* tokens per slot: 16 or 32                              */
    int32_t num_layers;       /* layers held by each pool (>= 1)                        */
    int64_t num_slots;        /* slots per layer                                        */
} sa_layout;

/* Device page table in CSR form (see the layout notes above). */
typedef struct sa_pages {
    const int32_t *indptr;    /* device [batch + 1]                                     */
    const int32_t *indices;   /* device [indptr[batch]] slot ids                        */
} sa_pages;

/* Create a context on HIP device `device` (must be gfx950).  The context owns
 * only plan buffers, pinned staging, split-KV scratch and an error flag.
 * Returns SA_ERR_DEVICE if the device is missing or not gfx950. */
sa_status sa_create(int device, sa_ctx **out);

/* Release a context (waits for the device first).  NULL is ignored. */
void sa_destroy(sa_ctx *ctx);

/* Static description of a status code. */
const char *sa_status_string(sa_status status);

/* Message of the most recent failing call on this thread ("" if none). */
const char *sa_last_error(void);

/*
 * sa_reserve — size the context's buffers ahead of time, so that later calls
 * whose plans fit them allocate no device or pinned memory (for example
 * before a timed loop or a serving loop).  plan_bytes: capacity of each call
 * kind's device plan buffer and of each pinned staging buffer; an attention
 * call's plan takes about 40 bytes per work item (one per sequence, KV head
 * and 128 packed query rows, and per key-range part of a split item) plus
 * 16 bytes per sequence, 24 per split item and 768 of alignment; a splice's
 * about 24 bytes per surviving page plus 16 per sequence.  split_bytes:
 * capacity of the split-KV partials, 128 * 129 * 4 bytes per key-range part.
 * Buffers only grow; outgrown ones are kept until sa_destroy.
 * Errors: SA_ERR_NULL (context), SA_ERR_SHAPE (negative size), SA_ERR_HIP.
 */
sa_status sa_reserve(sa_ctx *ctx, int64_t plan_bytes, int64_t split_bytes);

/*
 * sa_attn_plan_stats — the shape of the attention launch sa_segment_prefill_attn
 * would make for these lengths on a GPU with num_cu compute units (host only:
 * no context, no GPU), for latency models of a batch (paper Sec. 4, Eq. 1
 * models a batch from its decode and prefill work; how the work falls onto
 * the chip's workgroup slots adds to that).  out[0]: workgroups; out[1]:
 * key-range parts of split items (when > 0, a partial-merge launch follows);
 * out[2]: 64-key tiles over all items; out[3]: makespan in tiles when the
 * items are taken in launch order by whichever of the 2 x num_cu workgroup
 * slots frees first (a decode item's tiles count a quarter: its four waves
 * split them).  Errors: those of sa_segment_prefill_attn's shape checks;
 * SA_ERR_NULL for a NULL out; SA_ERR_SHAPE for num_cu < 1.
 */
sa_status sa_attn_plan_stats(const sa_layout *layout, int32_t batch, const int32_t *h_q_len,
                             const int32_t *h_kv_len, int32_t num_cu, int64_t *out);

/* Wait for `stream`, then report SA_ERR_RANGE if any kernel of this context
 * met an out-of-range page id or slot since the last check (and clear it). */
sa_status sa_sync_check(sa_ctx *ctx, void *stream);

/*
 * sa_kv_append — store a segment's new K/V rows in the cache (paper Sec. 3.2:
 * the lookahead transform builds KV on the transformed prefix).
 *
 * For each sequence b, new token t (0 <= t < h_new_len[b]) goes to logical
 * position h_start[b] + t of layer `layer`: slot
 * pages.indices[pages.indptr[b] + (h_start[b] + t) / page_size], row
 * (h_start[b] + t) % page_size.  Rows are copied bit for bit; nothing else in
 * the pools changes.  k_new / v_new hold the rows of all sequences back to
 * back ([sum new_len][Hkv][128]).  A sequence with h_new_len[b] == 0 is a
 * no-op.  The page list of b must cover the written positions.
 *
 * Errors: SA_ERR_SHAPE (batch < 1, negative start or length, layer outside
 * [0, num_layers)), SA_ERR_UNSUPPORTED, SA_ERR_NULL, SA_ERR_ALIGN, SA_ERR_HIP.
 */
sa_status sa_kv_append(sa_ctx *ctx, const sa_layout *layout, int32_t layer,
                       void *k_pool, void *v_pool,
                       const void *k_new, const void *v_new,
                       int32_t batch, const int32_t *h_start, const int32_t *h_new_len,
                       sa_pages pages, void *stream);

/*
 * sa_kv_assemble — commit splice into a replacement cache (paper Sec. 3.2
 * commit; Sec. 3.4 keep-recent-K drops an interior run of turns).
 *
 * Sequence b's source cache holds h_src_len[b] tokens on the pages of `src`.
 * Its surviving pages are the [begin, end) logical page spans
 * h_keep_spans[2*s], h_keep_spans[2*s+1] for s in h_keep_indptr[b] ..
 * h_keep_indptr[b+1]-1 (ascending, disjoint, non-empty, within the source
 * pages).  The replacement cache of b is those pages in order, renumbered
 * from 0, followed by enough new pages for h_reserve[b] more tokens:
 *   kept_b  = tokens on the surviving pages   (returned in h_dst_len[b])
 *   pages_b = ceil((kept_b + h_reserve[b]) / page_size)
 * Destination slots are taken from the front of the device free list
 * d_fresh[0 .. num_fresh), sequence after sequence.  Every surviving page is
 * copied whole (all page_size rows, every KV head, every layer) from its
 * source slot to its destination slot; reserved pages are left untouched.
 * The destination page table is written to d_dst_indptr[batch + 1] and
 * d_dst_indices[sum pages_b] (capacity dst_capacity entries).
 *
 * k_dst / v_dst may be the same pools as k_src / v_src.  Fresh slots must not
 * be surviving source slots of this call (the copy reads and writes in
 * parallel) and must not repeat; nothing checks this on the hot path
 * (SA_DEBUG=1 does, see the conventions above).
 *
 * Errors: SA_ERR_SHAPE, SA_ERR_RANGE (bad span), SA_ERR_NO_PAGES (free list
 * or dst_capacity too small), SA_ERR_UNSUPPORTED, SA_ERR_NULL, SA_ERR_ALIGN,
 * SA_ERR_HIP.
 */
sa_status sa_kv_assemble(sa_ctx *ctx, const sa_layout *layout,
                         const void *k_src, const void *v_src, void *k_dst, void *v_dst,
                         int32_t batch, const int32_t *h_src_len,
                         const int32_t *h_keep_indptr, const int32_t *h_keep_spans,
                         const int32_t *h_reserve,
                         sa_pages src, const int32_t *d_fresh, int32_t num_fresh,
                         int32_t *d_dst_indptr, int32_t *d_dst_indices, int32_t dst_capacity,
                         int32_t *h_dst_len, void *stream);

/*
 * sa_kv_assemble_append — sa_kv_assemble followed by the segment's
 * sa_kv_append, in one launch (paper Sec. 3.2: the transformed KV is the
 * spliced prefix plus the segment's rows).
 *
 * Arguments and results of sa_kv_assemble, plus: layer, the layer whose new
 * rows are written; k_new / v_new, bf16 [sum h_new_len][num_kv_heads][head_dim];
 * h_new_len[b] (host), the new tokens of sequence b, which go to logical
 * positions h_dst_len[b] .. h_dst_len[b] + h_new_len[b] - 1 of its
 * replacement cache (they must fit its pages: kept + new <= pages_b *
 * page_size).  The pools end exactly as after the two calls in sequence: the
 * rows of a partial last surviving page that the segment fills come from the
 * new rows, the rest of that page from its source.
 *
 * Errors: those of sa_kv_assemble, and SA_ERR_SHAPE for a bad layer or new
 * tokens that do not fit, SA_ERR_NULL for NULL new rows or h_new_len.
 */
sa_status sa_kv_assemble_append(sa_ctx *ctx, const sa_layout *layout,
                                const void *k_src, const void *v_src, void *k_dst, void *v_dst,
                                int32_t batch, const int32_t *h_src_len,
                                const int32_t *h_keep_indptr, const int32_t *h_keep_spans,
                                const int32_t *h_reserve,
                                sa_pages src, const int32_t *d_fresh, int32_t num_fresh,
                                int32_t *d_dst_indptr, int32_t *d_dst_indices, int32_t dst_capacity,
                                int32_t *h_dst_len, int32_t layer, const void *k_new,
                                const void *v_new, const int32_t *h_new_len, void *stream);

/*
 * sa_kv_splice_alias — zero-copy form of the commit splice (paper Sec. 3.2
 * commit, Sec. 3.4 keep-recent-K), for callers whose surviving pages may stay
 * where they are.
 *
 * Same spans, lengths, free list and outputs as sa_kv_assemble, but no page
 * is copied: the destination table of sequence b lists the SOURCE slots of its
 * surviving pages, in order, followed by fresh slots -- taken from the front of
 * d_fresh, sequence after sequence -- for the pages that h_reserve[b] more
 * tokens need beyond the surviving ones (so the free list is consumed only by
 * reserved pages).  The surviving pages are then shared between the source and
 * the destination tables: an append into the last surviving page (when it is
 * partial) writes into the source slot, past the source's own length.
 *
 * Errors: as sa_kv_assemble (d_fresh may be NULL when no page is reserved).
 * A missing source page or a source slot outside [0, num_slots) is latched in
 * the device flag that sa_sync_check reports (a missing page's entry is -1).
 */
sa_status sa_kv_splice_alias(sa_ctx *ctx, const sa_layout *layout, int32_t batch,
                             const int32_t *h_src_len, const int32_t *h_keep_indptr,
                             const int32_t *h_keep_spans, const int32_t *h_reserve,
                             sa_pages src, const int32_t *d_fresh, int32_t num_fresh,
                             int32_t *d_dst_indptr, int32_t *d_dst_indices, int32_t dst_capacity,
                             int32_t *h_dst_len, void *stream);

/*
 * sa_segment_prefill_attn — causal grouped-query attention of each
 * sequence's last h_q_len[b] tokens over its h_kv_len[b] cached tokens
 * (paper Sec. 4, prefill-attention term; decode rows are the q_len = 1 case of
 * the decode-attention term).
 *
 * With prefix_b = h_kv_len[b] - h_q_len[b], segment row i of query head h
 * attends keys 0 .. prefix_b + i of KV head h / (Hq / Hkv) in layer `layer`:
 *   O = softmax(softmax_scale * q . K^T) V,   LSE = log(sum exp(scale * q . k))
 * The segment's own K/V must already be in the cache (sa_kv_append).  Output
 * rows are bf16 (round to nearest even); `lse` may be NULL.  Sequences with
 * h_q_len[b] == 0 are skipped.  Arithmetic: bf16 MFMA products with fp32
 * accumulation, fp32 online softmax, probabilities rounded to bf16 before the
 * PV product.  The scale is applied to each fp32 score (with log2(e)) before
 * the exponential; a row's exponent offset moves only when its max grows by
 * more than 2^8, and the bf16 rounding of the probability of every key that
 * was its row's largest when it arrived is carried into the normaliser of the
 * output (not into the LSE), so a dominant key's weight comes out as its
 * exact share.  After sa_set_exact_scale(ctx, 0) the kernel instead
 * multiplies each query row by softmax_scale * log2(e) once and rounds it to
 * bf16 (faster; moves a row's scaled scores by up to
 * 2^-8 * sum_d |scale log2(e) q_d k_d| in log2 units).
 *
 * Errors: SA_ERR_SHAPE (0 <= q_len <= kv_len violated, bad batch or layer,
 * softmax_scale not finite and positive),
 * SA_ERR_UNSUPPORTED, SA_ERR_NULL, SA_ERR_ALIGN, SA_ERR_HIP.
 */
sa_status sa_segment_prefill_attn(sa_ctx *ctx, const sa_layout *layout, int32_t layer,
                                  const void *q, const void *k_pool, const void *v_pool,
                                  int32_t batch, const int32_t *h_q_len, const int32_t *h_kv_len,
                                  sa_pages pages, float softmax_scale,
                                  void *o, float *lse, void *stream);

/*
 * sa_segment_prefill_attn_noalloc — sa_segment_prefill_attn for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same arguments, same results (bit
 * for bit as long as its split-KV partials fit, see below), but it calls no
 * hipMalloc, hipFree or other allocating HIP routine (the host planner uses
 * only ordinary C++ heap memory): the launch's plan and its split-KV partials
 * live in one fixed device array of 32 MiB per GPU, a file-scope
 * `static __device__` array that each GPU the library runs on holds until
 * the process ends; the plan reaches it through pinned staging the context
 * allocated at sa_create.  Limits: the plan (about 40 bytes per work item, a
 * work item per sequence, KV head and 128 packed query rows) must fit 2 MiB,
 * else SA_ERR_SHAPE before anything is enqueued; the partials get the other
 * 30 MiB (476 key-range parts of 128 rows), and a launch that would split
 * into more parts is split more coarsely instead.  Every call on one GPU uses
 * that GPU's array, whichever context makes it, and leaves the last call's
 * contents there: calls that overlap in time on one GPU (two streams, two
 * contexts) race, so order them.  The call may wait on the host for the
 * previous plan copy of the same context to finish.
 * Errors: those of sa_segment_prefill_attn.
 */
sa_status sa_segment_prefill_attn_noalloc(sa_ctx *ctx, const sa_layout *layout, int32_t layer,
                                          const void *q, const void *k_pool, const void *v_pool,
                                          int32_t batch, const int32_t *h_q_len, const int32_t *h_kv_len,
                                          sa_pages pages, float softmax_scale,
                                          void *o, float *lse, void *stream);

/*
 * sa_set_exact_scale — how later attention calls on this context apply
 * softmax_scale.  enable != 0 (the default) multiplies each fp32 score by it
 * (with log2(e)) before the exponential: the only roundings are those of the
 * probabilities to bf16 before the PV product and of the output.  enable == 0
 * is a fast mode that folds the scale into the query rows, rounded to bf16
 * once per row, which saves one fma per score and moves the scores by at most
 * 2^-8 * sum_d |scale log2(e) q_d k_d| (log2 units) -- of the order of the
 * error bf16 query and key rows already carry, but large when the logits
 * are.  Applies to the default kernel; SA_ATTN_VARIANT=1 always scales in
 * fp32, SA_ATTN_VARIANT=2 never.  Errors: SA_ERR_NULL for a NULL context.
 */
sa_status sa_set_exact_scale(sa_ctx *ctx, int32_t enable);

/*
 * sa_set_fused_append — how later sa_segment_prefill_attn_append calls on
 * this context write the segment's rows.  enable != 0: inside the attention
 * launch, which reads the segment's keys from k_new / v_new; enable == 0 (the
 * default): an append launch (sa_kv_append) and then the attention.  Both
 * forms leave the same pool; their outputs are equal bit for bit when every
 * prefix length is a multiple of 4 and no request has at most 32 query rows,
 * and otherwise both are held to the same tolerance.
 * Errors: SA_ERR_NULL for a NULL context.
 */
sa_status sa_set_fused_append(sa_ctx *ctx, int32_t enable);

/*
 * sa_set_kernel_events — timing hook for measurement.  While set for `which`,
 * every kernel of that kind this context launches is launched by
 * hipExtLaunchKernelGGL with start_event and stop_event (hipEvent_t handles
 * the caller created with timing enabled), which binds both events to that
 * kernel, so their elapsed time is the kernel's execution on the device
 * rather than that of the call (events recorded around a call also span the
 * dispatch gap, several microseconds).  Kinds:
 *   SA_TIMED_ATTN   the attention kernel of sa_segment_prefill_attn and
 *                   sa_segment_prefill_attn_append (not the partial merge
 *                   that follows a launch split by key range)
 *   SA_TIMED_PAGES  the page kernel of sa_kv_append, sa_kv_assemble,
 *                   sa_kv_assemble_append, sa_kv_splice_alias and the append
 *                   launch of sa_segment_prefill_attn_append
 * A later launch of the same kind re-binds the same events.  Both NULL clears
 * the hook; the events stay owned by the caller and must outlive the launches.
 * Errors: SA_ERR_NULL for a NULL context or one event without the other,
 * SA_ERR_SHAPE for an unknown kind.
 */
#define SA_TIMED_ATTN 0
#define SA_TIMED_PAGES 1
sa_status sa_set_kernel_events(sa_ctx *ctx, int32_t which, void *start_event, void *stop_event);

/*
 * sa_set_block_clock — per-workgroup timestamps for measurement (which work of
 * a mixed decode + prefill launch ends when; paper Sec. 4 and Alg. 2 batch
 * decode requests with prefill chunks).  While set, each launch of the default
 * attention kernel writes, for every workgroup w, four uint64 words at
 * d_buf[4w]: the device's constant-rate wall clock (s_memrealtime) when w
 * started and when all its output stores were done; then its work item: word
 * 2 holds the sequence index in bits 0-31, the KV head in bits 32-47 and the
 * item's first key tile (of 64 keys) modulo 2^16 in bits 48-63; word 3 holds
 * that sequence's q_len in bits 0-31 (1: a decode row; 0 for a workgroup with
 * no work, which the planner adds to even out the XCDs) and the item's first
 * packed query row in bits 32-63.  The launch has one workgroup per
 * work item, at most max_blocks of them, else it fails with SA_ERR_SHAPE
 * before launching.  d_buf: device memory of 32 * max_blocks bytes, 8-byte
 * aligned, owned by the caller; the words of one launch are overwritten by
 * the next.  clock_khz (nullable, host): receives the clock's rate in kHz.
 * NULL, 0 clears.  The other attention kernels (SA_ATTN_VARIANT 1, 2) write
 * nothing.  Errors: SA_ERR_NULL (context), SA_ERR_SHAPE, SA_ERR_ALIGN,
 * SA_ERR_HIP.
 */
sa_status sa_set_block_clock(sa_ctx *ctx, void *d_buf, int64_t max_blocks, int64_t *clock_khz);

/*
 * sa_set_xcd_weights — relative speeds of the chip's 8 XCDs (workgroup i of a
 * launch runs on XCD i % 8) for the attention planner.  The XCDs of one
 * MI355X do not run equally fast under a long MFMA-bound launch (their clocks
 * differ by several percent), and a launch ends with its slowest XCD.  With
 * speeds set, the planner, when it places the work items of each KV head on
 * one XCD, evens out key tiles per unit of speed across the XCDs of a launch
 * of at most two rounds of workgroups: it pairs the XCDs by speed (slowest
 * with fastest, and so on) and, within each pair, swaps the longest item of
 * the XCD whose busiest CU is the more loaded for the shortest item of the
 * other (every XCD keeps its number of items; a moved item reads its KV
 * head's K/V through the other XCD's L2).  Launches of more rounds are placed
 * as without speeds.  Results are
 * unchanged bit for bit (a work item's arithmetic does not depend on where it
 * runs).  h_speed: host float[8], each finite and > 0 (only ratios matter),
 * e.g. the inverse of each XCD's mean workgroup time from sa_set_block_clock
 * on a launch with equal work per XCD; NULL resets to equal speeds.
 * Errors: SA_ERR_NULL (context), SA_ERR_SHAPE.
 */
sa_status sa_set_xcd_weights(sa_ctx *ctx, const float *h_speed);

/*
 * sa_segment_prefill_attn_append — the segment's append and its attention in
 * one call: each sequence's h_q_len[b] new K/V rows are written to its
 * logical positions h_kv_len[b] - h_q_len[b] .. h_kv_len[b] - 1 (as
 * sa_kv_append with start = kv_len - q_len), then the attention is computed
 * exactly as sa_segment_prefill_attn does over the cache that results (paper
 * Sec. 3.2: the lookahead builds the segment's KV on the transformed prefix).
 * k_new / v_new: bf16 [sum h_q_len][num_kv_heads][head_dim], token-major like
 * q; the pools are written.  The pages for the new rows must already be in
 * the table (sa_kv_assemble's reserve).  By default this is the append
 * kernel followed by the attention kernel on `stream`.  With fusion switched
 * on (sa_set_fused_append) it is one launch of the default attention kernel:
 * every workgroup reads the segment's keys and values from k_new / v_new, not
 * from their pages, and the first key-range part of each 128-row tile writes
 * the rows of the tokens whose first query row lies in that tile, so the rows
 * are written once and no workgroup waits on another (a request of at most
 * 32 query rows writes its own rows and reads them back).  The fused form
 * falls back to the two launches for the other kernel variants
 * (SA_ATTN_VARIANT), when a layer's pool spans 2^31 bytes or more, or when
 * k_new does.  The rows written must not be
 * rows that another sequence of the call reads as part of its prefix (as with
 * the two launches, whose order would otherwise decide what it reads).
 *
 * Errors: those of sa_segment_prefill_attn; SA_ERR_NULL for NULL new rows
 * (when any q_len > 0), SA_ERR_ALIGN for new rows not 16-byte aligned.  A
 * missing or out-of-range page of a new row raises the device error flag
 * (reported by sa_sync_check) and that row is not written.
 */
sa_status sa_segment_prefill_attn_append(sa_ctx *ctx, const sa_layout *layout, int32_t layer,
                                         const void *q, void *k_pool, void *v_pool,
                                         const void *k_new, const void *v_new, int32_t batch,
                                         const int32_t *h_q_len, const int32_t *h_kv_len,
                                         sa_pages pages, float softmax_scale, void *o, float *lse,
                                         void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SA_H */
