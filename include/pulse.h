/*
 * pulse.h -- C ABI of the MI355X (gfx950) sparse-KV decode hot path.
 *
 * One layer-step of I/O-centric sparse KV-cache offloading (PulseInfer,
 * arXiv 2609.34555): score the current query against per-block key digests
 * of one KV head, select one top-k block set shared by all KV heads
 * (SoloHead, Sec. 4.4.1), take the set difference against the GPU-resident
 * hot set, recall the missing blocks from pinned host DRAM into a GPU slot
 * pool while updating the block table (Sec. 2.2, Sec. 4.4.2), and run sparse
 * GQA decode attention over the selected blocks.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Ownership.  The caller owns every buffer.  The compute entry points never
 *   allocate or free memory, never synchronise the host and keep no global
 *   state; calls on disjoint buffers may run concurrently.
 * Asynchrony.  Every compute call only enqueues work on `stream` and returns.
 *   The return value reports errors detectable on the host before launch
 *   (null pointers, unsupported shapes, workspace too small) and launch
 *   failures (PULSE_ERR_HIP).  On any non-OK return nothing was enqueued.
 * Device-detected errors.  Conditions that depend on device data (pool
 *   exhaustion, a selection larger than k_max, an index outside its buffer)
 *   are reported by writing the code into `*dev_status` (a device int32 that
 *   the caller zeroes; the first error written wins, OK is never written).
 *   Every such condition is checked before the memory access it guards, so a
 *   bad index never turns into an out-of-bounds access.
 * Element types.  K, V and queries are fp16 or bf16 (pulse_dtype); they are
 *   passed as raw 16-bit element buffers.  Scores, outputs and LSE are fp32.
 * Indices.  Block and slot indices are int32; block offsets are int64.
 * Inputs must be finite.
 *
 * Supported shapes: head_dim 128; block_size 16, 32 or 64; num_q_heads a
 * multiple of num_kv_heads with G = num_q_heads / num_kv_heads in [1, 16].
 *
 * KV block layout (host store and slot pool alike).  One block holds all KV
 * heads of bs consecutive tokens, K first, then V:
 *   K(h, t, c) at element ((0 * Hkv + h) * bs + t) * d + c      token-major
 *   V(h, t, c) at element Hkv*bs*d + (h * d + c) * bs + t       channel-major
 * so a block is U = 2 * Hkv * bs * d * 2 bytes (64 KiB at Hkv 8, bs 16).
 * Tokens past the end of a context inside its last block must be zero.
 * Requests are ragged: request r owns n_r = ceil(ctx_len[r] / bs) blocks,
 * its global blocks are blk_off[r] .. blk_off[r+1]-1 (blk_off[0] = 0).
 */
#ifndef PULSE_H
#define PULSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PULSE_API __attribute__((visibility("default")))

typedef struct ihipStream_t* pulse_stream_t; /* a hipStream_t; NULL = default stream */

typedef enum {
    PULSE_OK = 0,
    PULSE_ERR_INVALID_ARG = 1,     /* host-detected: null pointer, negative size, bad index arg */
    PULSE_ERR_UNSUPPORTED = 2,     /* host-detected: shape or dtype outside the supported set */
    PULSE_ERR_WORKSPACE = 3,       /* host-detected: ws_bytes below pulse_workspace_bytes() */
    PULSE_ERR_POOL_EXHAUSTED = 4,  /* device-detected: more missing blocks than free slots */
    PULSE_ERR_SELECT_OVERFLOW = 5, /* device-detected: forced + k_mid blocks exceed k_max */
    PULSE_ERR_HIP = 6,             /* a HIP launch or runtime call failed */
    PULSE_ERR_BAD_INDEX = 7,       /* device-detected: block/slot index outside its buffer,
                                      or a selection list not strictly ascending */
    PULSE_ERR_TIMEOUT = 8          /* host-side wait expired (gather-scatter engine) */
} pulse_status;

typedef enum { PULSE_F16 = 0, PULSE_BF16 = 1 } pulse_dtype;

typedef struct {
    int32_t num_q_heads;  /* Hq */
    int32_t num_kv_heads; /* Hkv */
    int32_t head_dim;     /* d, must be 128 */
    int32_t block_size;   /* bs, tokens per KV block: 16, 32 or 64 */
    int32_t dtype;        /* pulse_dtype of K, V and q */
} pulse_shape;

/* Device-resident statistics written by the recall (device memory). */
typedef struct {
    int32_t n_missing; /* blocks recalled (on pool exhaustion or a bad free slot: blocks
                          that would be; on a malformed selection: 0) */
    int32_t n_runs;    /* maximal runs of consecutive missing block indices (0 on a
                          malformed selection) */
    int64_t bytes;     /* bytes copied host -> slot pool (0 on any device error) */
} pulse_recall_stats;

/* Human-readable name of a status code (static string). */
PULSE_API const char* pulse_status_string(pulse_status s);

/* Bytes of one KV block of `shape` (U above); 0 if the shape is unsupported. */
PULSE_API size_t pulse_block_bytes(const pulse_shape* shape);

/*
 * Workspace bytes needed by every compute entry point for a batch of B
 * requests, at most k_max selected blocks per request and total_blocks
 * blocks in all (sum of n_r).  One workspace of this size serves any call
 * with the same or smaller arguments, including pulse_decode_layer.
 * Returns 0 for an unsupported shape or negative sizes.
 */
PULSE_API size_t pulse_workspace_bytes(const pulse_shape* shape, int32_t B, int32_t k_max, int64_t total_blocks);

/*
 * a1. Per-block key digest of one KV head (Sec. 2.1: compact per-block
 * digests in the style of Quest; Sec. 4.4.1: SoloHead keeps digests for one
 * KV head per layer only).  For every block b of request r and channel c:
 *   digests[b][0][c] = min over valid tokens t of K(kv_head, t, c)
 *   digests[b][1][c] = max over valid tokens t of K(kv_head, t, c)
 * exactly, in the KV dtype (-0 orders below +0).
 *   kv           [total_blocks][block] elements; device memory or pinned,
 *                host-mapped memory (the kernel reads it directly)
 *   blk_off      device int64 [B+1];   ctx_len  device int32 [B]
 *   total_blocks = blk_off[B] (host copy of the value, sizes the grid)
 *   digests      device, [total_blocks][2][head_dim] elements, written
 * Errors: host-detected only (a block whose request cannot be found is
 * skipped and reported as PULSE_ERR_BAD_INDEX through dev_status if given;
 * dev_status may be NULL).
 */
PULSE_API pulse_status pulse_build_digests(const pulse_shape* shape, const void* kv, const int64_t* blk_off,
                                 const int32_t* ctx_len, int32_t B, int64_t total_blocks,
                                 int32_t kv_head, void* digests, int32_t* dev_status,
                                 pulse_stream_t stream);

/*
 * a2 + a3. SoloHead top-k block selection (Sec. 4.4.1; budget split into
 * sink, local and middle tokens, Sec. 5 setup; sink and local blocks stay
 * resident, Sec. 4.2).  For request r with n_r blocks:
 *   score[b] = (1/G) * sum_{g<G} sum_c max(q[r][h*G+g][c] * mn[b][c],
 *                                          q[r][h*G+g][c] * mx[b][c])
 *   with h = solo_kv_head, computed in fp32;
 *   forced  = blocks j < n_sink_blocks and j >= n_r - n_local_blocks;
 *   middle  = the other blocks; k' = min(max(k_mid[r], 0), #middle);
 *   chosen  = the k' middle blocks of highest score, equal scores taken in
 *             ascending block order;
 *   sel_idx[r][0 .. sel_cnt[r]) = forced U chosen, ascending; the rest -1.
 *   q            device [B][Hq][d] elements
 *   digests      device [total_blocks][2][d] elements of solo_kv_head
 *   k_mid        device int32 [B] middle-block budget per request
 *   sel_idx      device int32 [B][k_max], written;  sel_cnt device int32 [B]
 *   scores       optional device float [total_blocks]: if non-NULL receives
 *                the scores of middle blocks (forced entries are left as is)
 * A request whose selection would exceed k_max gets sel_cnt = 0 and
 * PULSE_ERR_SELECT_OVERFLOW in *dev_status (dev_status must be non-NULL).
 */
PULSE_API pulse_status pulse_select_solohead(const pulse_shape* shape, const void* q, const void* digests,
                                   const int64_t* blk_off, int32_t B, int64_t total_blocks,
                                   int32_t solo_kv_head, const int32_t* k_mid, int32_t n_sink_blocks,
                                   int32_t n_local_blocks, int32_t k_max, int32_t* sel_idx,
                                   int32_t* sel_cnt, float* scores, int32_t* dev_status, void* ws,
                                   size_t ws_bytes, pulse_stream_t stream);

/*
 * a9. Headwise selection, the baseline SoloHead replaces (Sec. 3.4: every KV
 * head selecting its own blocks fragments recall into per-head transfers;
 * Sec. 4.4.1 "headwise" strategy).  Every KV head h scores and selects with
 * its own digests by the rule of pulse_select_solohead, and its selection is
 * diffed against the shared block table: each missing (head, block) pair is
 * one transfer of that head's K and V (U / Hkv bytes).
 *   head_digests [Hkv][total_blocks][2][d] elements (pulse_build_digests per head)
 *   sel_idx [Hkv][B][k_max], sel_cnt [Hkv][B]        device int32, written
 *   miss_cnt [Hkv][B]  missing blocks per (head, request), written
 *   run_cnt  [Hkv][B]  runs of consecutive missing blocks per (head, request)
 *   ws       pulse_headwise_workspace_bytes() bytes
 * Nothing is recalled and the table is not changed.  Errors as for
 * pulse_select_solohead (block indices beyond max_blocks -> BAD_INDEX).
 */
PULSE_API size_t pulse_headwise_workspace_bytes(const pulse_shape* shape, int32_t B, int32_t k_max,
                                                int64_t total_blocks);
PULSE_API pulse_status pulse_select_headwise(const pulse_shape* shape, const void* q, const void* head_digests,
                                             const int64_t* blk_off, int32_t B, int64_t total_blocks,
                                             const int32_t* k_mid, int32_t n_sink_blocks, int32_t n_local_blocks,
                                             int32_t k_max, const int32_t* block_table, int32_t max_blocks,
                                             int32_t n_slots, int32_t* sel_idx, int32_t* sel_cnt, int32_t* miss_cnt,
                                             int32_t* run_cnt, int32_t* dev_status, void* ws, size_t ws_bytes,
                                             pulse_stream_t stream);

/*
 * Step-end release of a recall: the hot set is fixed-size (Sec. 4.2: sink,
 * local and hot middle blocks stay resident; recalled blocks serve one layer
 * step), so after the step's attention the blocks the last recall mapped go
 * back to "not resident" (block_table entry -1) and their slots back to the
 * free list: *free_head -= stats.n_missing, then stats is cleared.  This is
 * the exact undo of that recall (allocation is LIFO from the free list), so
 * no allocation may happen between the recall and its release.  Reads the
 * recall plan (missing blocks per request) that the recall left in `ws`:
 * pass the workspace, B, k_max and total_blocks of the call that planned it
 * (pulse_decode_layer: its total_blocks; pulse_recall_gather and the
 * gather-scatter engine: 0).  A recall that moved no bytes (exhaustion, an
 * error, nothing missing) leaves nothing to undo; a second release is a no-op.
 * Stream-ordered, no host sync; inconsistent plans report BAD_INDEX in
 * dev_status.  pulse_decode_layer can instead release its predecessor's
 * recall itself (pulse_layer_args.release_previous).
 */
PULSE_API pulse_status pulse_release_recalled(const pulse_shape* shape, int32_t B, int32_t k_max,
                                              int64_t total_blocks, int32_t* block_table, int32_t max_blocks,
                                              int32_t* free_head, pulse_recall_stats* stats, int32_t* dev_status,
                                              void* ws, size_t ws_bytes, pulse_stream_t stream);

/*
 * Average selection (Sec. 4.4.1, the "average" strategy SoloHead is compared
 * with): every KV head h scores the blocks with its own digests
 * (head_digests[h], laid out as for pulse_select_headwise), the scores are
 * averaged over the KV heads, in fp32, heads summed in ascending order --
 * i.e. the mean over all query heads -- and one top-k on the average, with
 * the sink / local / tie rules of pulse_select_solohead, is shared by all
 * heads.
 *   scores   optional device float [total_blocks]: the averaged scores
 *            (forced blocks are not written); NULL keeps them in ws
 *   ws       pulse_average_workspace_bytes() bytes of device memory
 * Other arguments, outputs and errors as for pulse_select_solohead.
 */
PULSE_API size_t pulse_average_workspace_bytes(const pulse_shape* shape, int32_t B, int32_t k_max,
                                               int64_t total_blocks);
PULSE_API pulse_status pulse_select_average(const pulse_shape* shape, const void* q, const void* head_digests,
                                            const int64_t* blk_off, int32_t B, int64_t total_blocks,
                                            const int32_t* k_mid, int32_t n_sink_blocks, int32_t n_local_blocks,
                                            int32_t k_max, int32_t* sel_idx, int32_t* sel_cnt, float* scores,
                                            int32_t* dev_status, void* ws, size_t ws_bytes, pulse_stream_t stream);

/*
 * Middle Attention Mass (Eq. 2, Sec. 4.4.1), the offline calibration that
 * picks the solo head.  For query head q of request r, MAM_q is the softmax
 * mass of its full attention over the request's context that falls on the
 * middle blocks (all blocks except the first n_sink_blocks and the last
 * n_local_blocks, i.e. the blocks selection ranks); the KV head's MAM is the
 * mean of MAM_q over its G query heads:
 *   mam[r][h] = (1/G) sum_g exp(lse_middle(r, hG+g) - lse_all(r, hG+g)),
 * with lse the natural log-sum-exp of the logits q.k * sm_scale.  Computed
 * with the sparse attention kernel over every block and over the middle
 * blocks (fp32; no middle blocks -> 0).
 *   slot_pool / block_table  as for pulse_sparse_decode_attn; every block of
 *            every request must be resident (block_table[r][j] valid for
 *            j < ceil(ctx_len[r] / block_size) <= max_blocks), else
 *            PULSE_ERR_BAD_INDEX is reported in dev_status
 *   mam      device float [B][num_kv_heads], written
 *   ws       pulse_mam_workspace_bytes() bytes of device memory
 */
PULSE_API size_t pulse_mam_workspace_bytes(const pulse_shape* shape, int32_t B, int32_t max_blocks);
PULSE_API pulse_status pulse_mam(const pulse_shape* shape, const void* q, const void* slot_pool, int32_t n_slots,
                                 const int32_t* block_table, int32_t max_blocks, const int32_t* ctx_len, int32_t B,
                                 int32_t n_sink_blocks, int32_t n_local_blocks, float sm_scale, float* mam,
                                 int32_t* dev_status, void* ws, size_t ws_bytes, pulse_stream_t stream);

/*
 * Solo-head choice from MAM rows (host arrays, [rows][num_kv_heads], e.g. one
 * row per request or per calibration prompt): the KV head with the highest
 * summed MAM is the SoloHead (Sec. 4.4.1), the one with the lowest is the
 * "reversed" choice the paper uses as a control (Sec. 4.4.1, Table of
 * accuracy results); ties go to the lowest index.  Host-only.
 */
PULSE_API pulse_status pulse_pick_solo_heads(const float* mam, int32_t rows, int32_t num_kv_heads, int32_t* solo,
                                             int32_t* reversed);

/*
 * a4 + a5 + a6. Set difference, slot allocation and gather-scatter recall
 * (Sec. 2.2: B_recall = B_topk minus B_gpu, then copy from DRAM; Sec. 4.4.2:
 * scattered blocks move as coalesced transfers and land in the KV cache).
 *   missing = [(r, j) : r ascending, j = sel_idx[r][i] in listed order,
 *              block_table[r][j] == -1]
 *   the g-th missing block takes slot s = free_slots[*free_head + g];
 *   block_table[r][j] = s; slot_pool[s] = host_kv[blk_off[r] + j] (U bytes);
 *   *free_head += #missing; stats = {#missing, #runs, #missing * U}.
 * A run is a maximal stretch of listed missing blocks of one request whose
 * indices increase by one; runs are read from host memory as contiguous
 * streams.  The copy is done by GPU loads of the pinned host memory.
 *   host_kv      pinned, host-mapped [total_blocks][block] (hipHostMalloc
 *                with hipHostMallocMapped); read only
 *   sel_idx/sel_cnt  as produced by pulse_select_solohead (strictly
 *                ascending per request)
 *   block_table  device int32 [B][max_blocks], -1 = not resident; updated
 *   free_slots   device int32 [n_free];  free_head device int32, updated
 *   slot_pool    device [n_slots][block] elements; free slots are written
 *   stats        device pulse_recall_stats, written
 *   dev_status   device int32, required
 * If #missing > n_free - *free_head, PULSE_ERR_POOL_EXHAUSTED is reported and
 * the table, pool and free_head are left unchanged; likewise for any index
 * outside its buffer (PULSE_ERR_BAD_INDEX): a selection entry, a block_table
 * entry >= n_slots, *free_head outside [0, n_free], or any of the slots
 * free_slots[*free_head .. *free_head + #missing) outside [0, n_slots).  Every
 * slot is checked before anything is written, so on any of these errors no
 * table entry, pool byte or free_head changes and stats.bytes is 0.
 */
PULSE_API pulse_status pulse_recall_gather(const pulse_shape* shape, const void* host_kv, const int64_t* blk_off,
                                 int32_t B, const int32_t* sel_idx, const int32_t* sel_cnt, int32_t k_max,
                                 int32_t* block_table, int32_t max_blocks, const int32_t* free_slots,
                                 int32_t* free_head, int32_t n_free, void* slot_pool, int32_t n_slots,
                                 pulse_recall_stats* stats, int32_t* dev_status, void* ws,
                                 size_t ws_bytes, pulse_stream_t stream);

/*
 * The paper's own recall engine as a second recall path (Sec. 4.4.2:
 * gather the scattered blocks on the CPU into a contiguous pinned staging
 * buffer, move them with one large DMA, scatter them into the GPU KV cache
 * with a GPU kernel; Sec. 4.5: zero-sync submission -- the GPU writes the
 * selected indices and a ready flag into host-visible memory and a CPU
 * polling thread builds the recall task for I/O worker threads).
 *
 * pulse_gs_engine_create: one engine per device and shape.  Owns a pinned
 *   mailbox for up to max_blocks_per_call plan entries, two pinned and two
 *   device staging buffers of staging_blocks blocks each (batches alternate
 *   between them), a copy stream for the DMAs and a scatter stream, n_workers
 *   gather threads and a poller thread.
 *   Allocation happens here, never in the calls below.
 * pulse_gs_recall_submit: same arguments and results as
 *   pulse_recall_gather (set difference, allocation, table / free_head /
 *   stats updates on `stream`), but the bytes move through the engine.
 *   Returns at once with a sequence number; one call may be in flight per
 *   engine (a second submit before completion -> PULSE_ERR_INVALID_ARG).
 *   The pool slots are valid once the call has completed.
 * pulse_gs_recall_poll: non-blocking completion check (*done = 1 when the
 *   blocks are in the pool; returns that call's device-detected status).
 * pulse_gs_recall_wait: blocks up to timeout_ms; PULSE_ERR_TIMEOUT if the
 *   call has not completed.  No GPU stream waits on the host: the caller
 *   enqueues attention after completion (the semi-synchronous check of
 *   Sec. 4.2.2 is a poll at a layer boundary).
 * pulse_gs_last_timing: milliseconds of the last completed call: CPU gather,
 *   the DMA + scatter tail after the last gather, total (poller clock).
 */
typedef struct pulse_gs_engine pulse_gs_engine;
PULSE_API pulse_status pulse_gs_engine_create(const pulse_shape* shape, int32_t n_workers,
                                              int64_t max_blocks_per_call, int64_t staging_blocks,
                                              pulse_gs_engine** engine);
PULSE_API pulse_status pulse_gs_engine_destroy(pulse_gs_engine* engine);
PULSE_API pulse_status pulse_gs_recall_submit(pulse_gs_engine* engine, const void* host_kv, const int64_t* blk_off,
                                              int32_t B, const int32_t* sel_idx, const int32_t* sel_cnt,
                                              int32_t k_max, int32_t* block_table, int32_t max_blocks,
                                              const int32_t* free_slots, int32_t* free_head, int32_t n_free,
                                              void* slot_pool, int32_t n_slots, pulse_recall_stats* stats,
                                              int32_t* dev_status, void* ws, size_t ws_bytes, int64_t* seq,
                                              pulse_stream_t stream);
PULSE_API pulse_status pulse_gs_recall_poll(pulse_gs_engine* engine, int64_t seq, int32_t* done);
PULSE_API pulse_status pulse_gs_recall_wait(pulse_gs_engine* engine, int64_t seq, int32_t timeout_ms);
PULSE_API pulse_status pulse_gs_last_timing(pulse_gs_engine* engine, float* ms3);

/*
 * a7. Sparse GQA decode attention over the selected blocks (the attention
 * that follows recall, Sec. 2.2 and Sec. 4.2.1).  For request r and query
 * head hq, KV head h = hq / G:
 *   logit_t = sm_scale * q[r][hq] . K(h, t)   over the valid tokens t of the
 *             blocks sel_idx[r][0 .. sel_cnt[r]), read from
 *             slot_pool[block_table[r][j]]
 *   out[r][hq] = sum_t softmax(logit)_t V(h, t)      (fp32)
 *   lse[r][hq] = log sum_t exp(logit_t)              (fp32, optional)
 * An empty selection gives out = 0 and lse = -inf.  Products and sums are
 * accumulated in fp32.
 *   out          device float [B][Hq][d];  lse optional device float [B][Hq]
 *   dev_status   device int32, required (unresident block -> BAD_INDEX)
 */
PULSE_API pulse_status pulse_sparse_decode_attn(const pulse_shape* shape, const void* q, const void* slot_pool,
                                      int32_t n_slots, const int32_t* block_table, int32_t max_blocks,
                                      const int32_t* sel_idx, const int32_t* sel_cnt, int32_t k_max,
                                      const int32_t* ctx_len, int32_t B, float sm_scale, float* out,
                                      float* lse, int32_t* dev_status, void* ws, size_t ws_bytes,
                                      pulse_stream_t stream);

/*
 * Split-K workgroups per (request, KV head) that pulse_sparse_decode_attn,
 * and the attention of pulse_decode_layer, launch for a batch of B requests
 * with at most k_max selected blocks each (the split depends on B, Hkv, k_max
 * and bs only).  Above 1, a kernel that merges the workgroups' partials
 * follows the split-K kernel, and pulse_layer_args.attn_split_event marks the
 * end of the split-K kernel alone.  At 1, one workgroup covers each (request,
 * KV head) and writes out / lse itself: no merge kernel runs, so a caller that
 * asks for both attn_split_event and events[4] gets events[4] recorded as a
 * marker packet after the kernel.  Host function, no device work; 0 for an
 * unsupported shape, B < 1 or k_max < 1.
 */
PULSE_API int32_t pulse_attention_workgroups(const pulse_shape* shape, int32_t B, int32_t k_max);

/* All arguments of one layer-step (pulse_decode_layer).  Field meanings are
 * those of the entry points above. */
typedef struct {
    pulse_shape shape;
    int32_t B;
    int64_t total_blocks;
    const int32_t* ctx_len;   /* device [B] */
    const int64_t* blk_off;   /* device [B+1] */
    const void* q;            /* device [B][Hq][d] */
    const void* digests;      /* device [total_blocks][2][d] of solo_kv_head */
    int32_t solo_kv_head;
    const int32_t* k_mid;     /* device [B] */
    int32_t n_sink_blocks;
    int32_t n_local_blocks;
    int32_t k_max;
    int32_t* sel_idx;         /* device [B][k_max], written */
    int32_t* sel_cnt;         /* device [B], written */
    const void* host_kv;      /* pinned host-mapped store */
    int32_t* block_table;     /* device [B][max_blocks], updated */
    int32_t max_blocks;
    const int32_t* free_slots;/* device [n_free] */
    int32_t* free_head;       /* device, updated */
    int32_t n_free;
    void* slot_pool;          /* device [n_slots][block] */
    int32_t n_slots;
    pulse_recall_stats* stats;/* device, written */
    float sm_scale;
    float* out;               /* device [B][Hq][d] */
    float* lse;               /* device [B][Hq] or NULL */
    int32_t* dev_status;      /* device, required */
    void* ws;
    size_t ws_bytes;
    void* const* events;      /* optional host array of 5 hipEvent_t for stage timing:
                                 [0] start and [1] end of the scoring kernel, [2] start
                                 and [3] end of the recall copy kernel, [4] end of the
                                 attention (its last kernel).  They ride on the kernels'
                                 own launches (hipExtLaunchKernel start / stop events),
                                 so they add no marker packets to the stream; NULL =
                                 none, and a NULL entry is not recorded.  With no block
                                 to score, [0] and [1] are recorded as markers.  A step
                                 captured into a HIP graph is captured without them
                                 (events and attn_split_event NULL; that is the form
                                 whose replays are tested) */
    int32_t release_previous; /* nonzero: before selecting, undo the recall of the
                                 previous pulse_decode_layer made with these buffers
                                 (table entries back to -1, free_head rewound; the hot
                                 set stays fixed-size, Sec. 4.2), inside the scoring
                                 kernel instead of a launch of its own.  Only a recall
                                 that moved bytes (stats->bytes > 0) is undone; the
                                 statistics are left for this step's recall to
                                 overwrite.  A recall made by pulse_recall_gather or
                                 the engine is released with pulse_release_recalled.
                                 0: no release */
    void* attn_split_event;   /* optional hipEvent_t recorded at the completion of the
                                 split-K attention kernel, before the kernel that merges
                                 its workgroup partials (if any): the launch carries it
                                 as the kernel's stop event, so the split-K kernel can
                                 be timed alone without a marker of its own; NULL = not
                                 recorded */
} pulse_layer_args;

/*
 * a8. One decode layer-step: score + select (with the set difference folded
 * into the selection pass), allocation + recall, attention, all enqueued on
 * one stream with no host synchronisation (zero-sync submission, Sec. 4.5).
 * Results are those of the four calls above made in order.
 */
PULSE_API pulse_status pulse_decode_layer(const pulse_layer_args* args, pulse_stream_t stream);

/*
 * pulse_decode_layer for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * workspace comes from a static device array of PULSE_NOALLOC_SCRATCH_BYTES
 * that the library holds on each GPU it runs on until the process ends, so the
 * caller passes args->ws = NULL and args->ws_bytes = 0 (else
 * PULSE_ERR_INVALID_ARG) and still owns every input and output buffer.  A call
 * whose workspace (pulse_workspace_bytes(shape, B, k_max, total_blocks)) would
 * exceed that size returns PULSE_ERR_WORKSPACE and enqueues nothing.  The
 * first call on a device looks up that device's array (no allocation); a
 * failed lookup returns PULSE_ERR_HIP.  Results are those of
 * pulse_decode_layer with a workspace of its own.
 * Every call on one GPU shares that GPU's array and finds there what the last
 * call left: calls that overlap on one GPU (concurrent streams, threads) race
 * and must not be made.  Each call writes every workspace word it reads, except
 * release_previous, which reads the plan the previous call left: it is valid only
 * when the previous call on this GPU was pulse_decode_layer_noalloc with the same
 * B, k_max and total_blocks on the same table, free list and statistics.
 */
#define PULSE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
PULSE_API pulse_status pulse_decode_layer_noalloc(const pulse_layer_args* args, pulse_stream_t stream);

/* ---- Interruptible layer-wise scheduling (IRQ, Sec. 4.2) ---- */

/*
 * One decode layer of a normal batch (Sec. 4.2: short requests whose KV cache
 * stays in HBM): decode attention over every block of each request, as
 * pulse_sparse_decode_attn with every block selected, then a SwiGLU FFN on its
 * output:
 *   x = bf16(out) [B][D], D = num_q_heads * head_dim;
 *   [g | u] = x . w_gate_up^T  [B][2 d_ff];   h = silu(g) * u  [B][d_ff];
 *   y = h . w_down^T  [B][D]
 * (bf16 storage, fp32 accumulation; projections and norms are not modelled).
 * All pointers are device memory owned by the caller:
 *   w_gate_up bf16 [2 d_ff][D] (gate rows, then up rows); w_down bf16 [D][d_ff];
 *   x, gu, h, y bf16 scratch / output of the sizes above; out, lse as for
 *   pulse_sparse_decode_attn; ws pulse_workspace_bytes(shape, B, k_max, 0).
 * The GEMMs (the library's MFMA kernel) read 16-byte pieces of rows: d_ff must
 * be a multiple of 8 (else PULSE_ERR_UNSUPPORTED) and w_gate_up, w_down, x and
 * h 16-byte aligned (else PULSE_ERR_INVALID_ARG).
 */
typedef struct pulse_normal_layer {
    pulse_shape shape;
    int32_t B;
    const void* q;
    const void* slot_pool;
    int32_t n_slots;
    const int32_t* block_table;
    int32_t max_blocks;
    const int32_t* sel_idx;
    const int32_t* sel_cnt;
    int32_t k_max;
    const int32_t* ctx_len;
    float sm_scale;
    float* out;
    float* lse;
    void* ws;
    size_t ws_bytes;
    int32_t d_ff;
    const void* w_gate_up;
    const void* w_down;
    void* x;
    void* gu;
    void* h;
    void* y;
    int32_t* dev_status;
} pulse_normal_layer;

/* Completion-detection modes of pulse_irq_step (Sec. 4.2.2). */
enum {
    PULSE_IRQ_SEMI_SYNC = 0, /* wait for a normal layer's attention, then check (the paper's choice) */
    PULSE_IRQ_SYNC = 1,      /* wait for the whole normal layer, then check */
    PULSE_IRQ_ASYNC = 2,     /* never wait; check between enqueues, at most async_ahead layers queued */
    PULSE_IRQ_BLOCKING = 3   /* no interleaving: wait for each recall, then one normal layer */
};

typedef struct pulse_irq_stats {
    int64_t normal_layers;      /* normal-batch layers run during the step */
    int32_t offload_layers;     /* offload-batch layers completed */
    int32_t max_overlap_depth;  /* most normal layers run during one recall */
    double mean_overlap_depth;  /* normal layers per recall wait (Sec. 4.2.1's overlap depth m) */
    double wall_ms;             /* host wall time of the step, all work finished */
    double mean_stall_us;       /* GPU time from a layer's selection to its attention: the offload batch parked */
    double mean_resume_us;      /* gather kernel path: GPU time from a recall's completion to its attention */
    double mean_recall_us;      /* gather kernel path: GPU time of a recall (copy + completion signal) */
} pulse_irq_stats;

typedef struct pulse_irq pulse_irq;

/*
 * Scheduler state for two caller-owned streams (compute, I/O; default
 * priority): a pinned host-mapped completion flag and timing events.
 * Allocates; not for use inside stream capture.  Destroy synchronises both
 * streams.
 */
PULSE_API pulse_status pulse_irq_create(pulse_stream_t compute_stream, pulse_stream_t io_stream, pulse_irq** irq);
PULSE_API pulse_status pulse_irq_destroy(pulse_irq* irq);

/*
 * One decode step of an offload batch -- n_offload_layers chained layer-steps
 * (pulse_layer_args as for pulse_decode_layer, B >= 1, one per layer) --
 * interleaved at layer boundaries with a normal batch that cycles through its
 * n_normal_layers layers (Sec. 4.2.1).  Offload layer m: selection on the
 * compute stream; recall on the I/O stream, then a signal kernel writes the
 * layer's sequence number into the pinned flag; until the host sees it, the
 * host keeps enqueuing normal layers on the compute stream and checks the flag
 * at each normal layer boundary as `mode` says (ASYNC: at most async_ahead
 * normal layers queued); then the offload attention for layer m is enqueued
 * (after a stream wait on the recall) and layer m + 1 follows.  With `engine`
 * (a pulse_gs_engine for the offload layers' shape; an offload layer of
 * another shape -> PULSE_ERR_INVALID_ARG before any work) the recall goes
 * through the gather-scatter engine instead, submitted on the compute stream, and its
 * host-side completion is the flag; the gather kernel path stalls concurrent
 * kernels on MI355X while it reads host memory, the engine's DMA does not.
 * Results of the offload batch are those of pulse_decode_layer on each layer
 * (mean_resume_us / mean_recall_us are -1 with an engine).
 * overlap_depth (optional host int32 [n_offload_layers]) receives the normal
 * layers run during each recall; stats is filled (host).  Returns after both
 * streams (and, after an early exit, an engine call in flight) are drained.
 * A recall whose flag is not seen within 60 s ends the step with
 * PULSE_ERR_TIMEOUT (after draining); device-side errors are in the layers'
 * dev_status words.
 */
PULSE_API pulse_status pulse_irq_step(pulse_irq* irq, const pulse_layer_args* offload, int32_t n_offload_layers,
                                      const pulse_normal_layer* normal, int32_t n_normal_layers, int32_t mode,
                                      int32_t async_ahead, pulse_gs_engine* engine, int32_t* overlap_depth,
                                      pulse_irq_stats* stats);

/* ---- IO-Adaptive Offloading Admission (Sec. 4.3; host side) ---- */

typedef struct {
    int64_t gpu_budget_bytes;    /* GPU memory available to newly admitted requests */
    int64_t kv_bytes_per_token;  /* KV bytes of one token over all layers and KV heads */
    int64_t offload_tokens;      /* GPU-resident hot budget of an offloaded request (tokens) */
    int64_t offload_extra_bytes; /* further GPU bytes per offloaded request (digests, tables) */
    int32_t running_normal;      /* requests already in the normal batch */
    int32_t running_offload;     /* requests already in the offload batch */
    const double* grid_bo;       /* profiled offload-batch sizes, ascending [n_bo] */
    int32_t n_bo;
    const double* grid_bn;       /* profiled normal-batch sizes, ascending [n_bn] */
    int32_t n_bn;
    const double* grid_m;        /* overlap depth m at (grid_bo[i], grid_bn[j]): [n_bo][n_bn] */
} pulse_ioaa_params;

/*
 * Overlap depth m(B_o, B_n): bilinear interpolation of the profiled grid,
 * clamped at its edges (Sec. 4.3.2: m = ceil(t_io / t_layer), profiled on a
 * (B_o, B_n) grid and interpolated from the nearest points).  NaN on a bad grid.
 */
PULSE_API double pulse_overlap_depth(const pulse_ioaa_params* params, double b_o, double b_n);

/*
 * Admission of n waiting requests (Sec. 4.3.1): maximise Eq. 1,
 *   thr = m/(m+1) * B_n + 1/(m+1) * B_o   (thr = B_n when B_o = 0),
 * over assignments of each request to the normal batch (its whole KV cache,
 * lengths[i] * kv_bytes_per_token bytes) or the offload batch (offload_tokens
 * * kv_bytes_per_token + offload_extra_bytes), by a depth-first binary-tree
 * search over the requests longest first with two prunes: the memory budget,
 * and no offloading after a longer request went to the normal batch.  A request
 * that fits neither batch ends its path (it and all shorter ones wait).
 *   assign[i] = 0 wait, 1 normal, 2 offload (host array); *throughput = Eq. 1
 *   at the chosen assignment; *nodes_visited (optional) = tree nodes the search
 *   visits; *leaves_evaluated (optional) = complete assignments at which it
 *   evaluates Eq. 1 (the admissible ones; a root-to-leaf path of n requests
 *   alone passes n + 1 nodes, so this is the count comparable with the
 *   paper's nodes-visited figure).
 * Host-only; no GPU work.
 */
PULSE_API pulse_status pulse_ioaa_plan(const pulse_ioaa_params* params, const int64_t* lengths, int32_t n,
                                       int8_t* assign, double* throughput, int64_t* nodes_visited,
                                       int64_t* leaves_evaluated);

/* ---- measurement helpers (host side; not part of the compute path) ---- */

/*
 * Pinned host memory for the KV store: hipHostMalloc with hipHostMallocMapped
 * | hipHostMallocPortable, plus hipHostMallocCoherent when `coherent` is
 * non-zero (fine-grained) or hipHostMallocNonCoherent otherwise.  *host_ptr
 * is usable by CPU code and by GPU kernels.  Free with pulse_host_free.
 */
PULSE_API pulse_status pulse_host_alloc(size_t bytes, int32_t coherent, void** host_ptr);
PULSE_API pulse_status pulse_host_free(void* host_ptr);

/*
 * Per-block hipMemcpyAsync recall baseline (one DMA per unit, as the
 * threaded per-block copy that the paper's gather-scatter engine is compared
 * with, Sec. 4.4.2).  Copies n units of unit_bytes from
 * host_kv + src_units[i] * unit_bytes to pool + dst_units[i] * unit_bytes.
 * src_units / dst_units are HOST arrays.  Enqueued on `stream`.
 */
PULSE_API pulse_status pulse_baseline_memcpy_units(const void* host_kv, void* pool, const int64_t* src_units,
                                         const int64_t* dst_units, int32_t n, size_t unit_bytes,
                                         pulse_stream_t stream);

/*
 * Host-link probe: a streaming kernel that copies `bytes` (a multiple of
 * 16384) from pinned host memory to device memory with the load pattern of
 * the recall kernel.  Used to measure the link's achievable read bandwidth.
 */
PULSE_API pulse_status pulse_probe_host_read(const void* host_src, void* dev_dst, size_t bytes, pulse_stream_t stream);

/*
 * HBM read probe: a streaming kernel that reads `bytes` (a multiple of 16) of
 * device memory at `src` and folds them into one word per workgroup in
 * `sink` (device, pulse_probe_hbm_sink_bytes() bytes).  Timed over the byte
 * count of an HBM-bound kernel, it measures the read bandwidth the GPU
 * sustains at that size.  start_event / stop_event (optional hipEvent_t):
 * recorded at the kernel's start and end by its launch, as the layer-step's
 * stage events are, so both are timed the same way.
 */
PULSE_API pulse_status pulse_probe_hbm_read(const void* src, size_t bytes, void* sink, void* start_event,
                                            void* stop_event, pulse_stream_t stream);
PULSE_API size_t pulse_probe_hbm_sink_bytes(void);

/* Timing events for pulse_layer_args.events: n hipEvent_t handles written to
 * events[0..n); destroy with pulse_events_destroy. */
PULSE_API pulse_status pulse_events_create(int32_t n, void** events);
PULSE_API pulse_status pulse_events_destroy(int32_t n, void* const* events);
/* Milliseconds between two completed events (hipEventElapsedTime). */
PULSE_API pulse_status pulse_event_elapsed_ms(void* start, void* stop, float* ms);

#ifdef __cplusplus
}
#endif

#endif /* PULSE_H */
