/*
 * mw.h - C ABI of the MI355X (gfx950) paged grouped-query attention library
 * for prefill/decode multiplexing on split compute units.
 *
 * The paper's statement of the problem: prefill and decode run at the same
 * time on disjoint sets of compute units of one GPU (Sec. 2.4 and Sec. 3.2.1),
 * both phases read and extend one paged KV-cache pool kept in the GPU's shared
 * memory space (Sec. 2.4; PagedAttention in Related Work), and each launch's
 * latency feeds the scheduler's estimates (Sec. 3.3).  AMD GPUs give the
 * intra-process partition through CU-masked streams (Sec. 5, Discussion).
 * This header exposes exactly those pieces:
 *
 *   mw_kv_pool_*   paged K/V pool descriptor, host page allocator, KV append
 *   mw_partition_* two CU-masked HIP streams with disjoint compute units
 *   mw_prefill_attn causal prefill attention of new tokens over a cached prefix
 *   mw_decode_attn  decode attention, one query token per sequence
 *   mw_timing_*    per-call GPU timings (HIP events)
 *
 * Conventions shared by every call
 * --------------------------------
 * - Status: every call returns mw_status (0 = MW_OK, negative = error) and
 *   never throws across the ABI.  The text of the last error of the calling
 *   thread is returned by mw_last_error().
 * - Ownership: every device buffer (pools, block tables, Q, O, workspaces) is
 *   owned by the caller; the library never frees one.  Handles (pool
 *   metadata, partitions and their streams, timing events) are owned by the
 *   library and released by the matching *_destroy call.
 * - Streams: an mw_stream is a hipStream_t; NULL means the null stream of
 *   the current device.
 * - Asynchrony: attention and pool-write calls only enqueue work.  They do
 *   no host<->device copies (a copy would serialise the two partitions), so
 *   lengths are passed twice: a host copy for planning and validation and a
 *   device copy for the kernels.  The two copies must hold the same values.
 * - Data types: K, V, Q and O are bf16 (raw 16-bit patterns); scores,
 *   softmax and accumulation are fp32.  Only head_dim 128 and page size 16
 *   are supported (MW_ERR_UNSUPPORTED otherwise).
 * - Layouts:
 *     K and V pools : [num_pages][num_kv_heads][page_size][head_dim] bf16,
 *                     so one (page, kv head) block is 4 KiB contiguous.
 *     block tables  : int32 [rows][bt_stride], row-major; entry t/page_size
 *                     of a row is the page holding token t of that sequence
 *                     (slot t % page_size).
 *     Q and O       : [tokens][num_q_heads][head_dim] bf16.
 *   Query head h reads KV head h / (num_q_heads / num_kv_heads).
 * - Device-side page indices outside [0, num_pages) are never dereferenced:
 *   kernels treat such a page as zeros or as absent (results are then
 *   meaningless, but no memory outside the pool is touched).
 * - Asynchronous HIP faults surface as MW_ERR_HIP from the next call that
 *   synchronises (mw_timing_elapsed, mw_sync), with the HIP error text in
 *   mw_last_error().
 */
#ifndef MW_H
#define MW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t mw_status;
#define MW_OK 0
#define MW_ERR_INVALID_ARG (-1)  /* a bad argument; nothing was enqueued        */
#define MW_ERR_UNSUPPORTED (-2)  /* valid but not implemented (head_dim, page)  */
#define MW_ERR_OUT_OF_PAGES (-3) /* the host page allocator has too few pages   */
#define MW_ERR_HIP (-4)          /* the HIP runtime reported an error           */
#define MW_ERR_NOT_READY (-5)    /* a timing was read before it was recorded    */

typedef void *mw_stream; /* a hipStream_t */
typedef struct mw_timing mw_timing; /* per-call GPU timing events (see below) */

/* Text of the calling thread's last error ("" if none).  The pointer stays
 * valid until the thread's next failing call. */
const char *mw_last_error(void);

/* Library ABI version (increments on any signature change). */
int32_t mw_version(void);

/* Waits for all work on `stream` and reports any pending HIP error. */
mw_status mw_sync(mw_stream stream);

/* ------------------------------------------------------------------------
 * KV pool (Sec. 2.4: one KV-cache pool shared by both phases; paged as in
 * PagedAttention).  The device arrays belong to the caller; the handle holds
 * their addresses, the geometry, and a host free-list of page ids.
 * ---------------------------------------------------------------------- */
typedef struct mw_kv_pool mw_kv_pool;
typedef struct {
    int32_t num_pages;    /* pages in each of the K and V arrays (>= 1)      */
    int32_t page_size;    /* tokens per page; must be 16                     */
    int32_t num_kv_heads; /* >= 1                                            */
    int32_t head_dim;     /* must be 128                                     */
} mw_kv_pool_desc;

/* Registers caller-owned device arrays d_k_pages / d_v_pages, each
 * num_pages*num_kv_heads*page_size*head_dim bf16 elements, 16-byte aligned.
 * The free list starts as 0, 1, ..., num_pages-1. */
mw_status mw_kv_pool_create(const mw_kv_pool_desc *desc, void *d_k_pages, void *d_v_pages,
                            mw_kv_pool **out);
mw_status mw_kv_pool_destroy(mw_kv_pool *pool);
/* Replaces the free list by `perm` (n distinct page ids in [0, num_pages)),
 * popped front first.  Lets a caller deal pages in a random order. */
mw_status mw_kv_pool_set_free_order(mw_kv_pool *pool, const int32_t *perm, int32_t n);
/* Pops n_pages ids from the free list into host array pages_out.  Fails with
 * MW_ERR_OUT_OF_PAGES (taking nothing) if fewer are free. */
mw_status mw_kv_pool_alloc(mw_kv_pool *pool, int32_t n_pages, int32_t *pages_out);
/* Returns pages to the back of the free list.  A page already free, or out
 * of range, is MW_ERR_INVALID_ARG (and nothing is returned). */
mw_status mw_kv_pool_free(mw_kv_pool *pool, const int32_t *pages, int32_t n_pages);
mw_status mw_kv_pool_num_free(const mw_kv_pool *pool, int32_t *n_free);

/* KV append (Sec. 2.1: each step stores the new tokens' keys and values in
 * the cache).  For each sequence b < batch, copies the rows
 * d_k_new[d_qo_indptr[b] + i] and d_v_new[...] (each [num_kv_heads][head_dim]
 * bf16) for i < h_new_lens[b] into position d_start_pos[b] + i of the
 * sequence whose block-table row is b.  A pure bit copy.
 *   h_new_lens  host  [batch]   new tokens per sequence (>= 0)
 *   h_start_pos host  [batch]   first position written (>= 0); validated
 *                               against bt_stride*page_size
 *   d_qo_indptr device[batch+1] row offsets into d_k_new / d_v_new
 *   d_start_pos device[batch]   same values as h_start_pos
 *   d_block_table device [batch][bt_stride]
 * `timing` may be NULL. */
mw_status mw_kv_pool_write(const mw_kv_pool *pool, int32_t batch, const int32_t *h_new_lens,
                           const int32_t *h_start_pos, const int32_t *d_qo_indptr,
                           const int32_t *d_start_pos, const int32_t *d_block_table,
                           int32_t bt_stride, const void *d_k_new, const void *d_v_new,
                           mw_stream stream, mw_timing *timing);

/* Gathers tokens [0, n_tokens) of one sequence (block-table row
 * d_block_table[0 .. ceil(n_tokens/page_size))) into contiguous
 * [n_tokens][num_kv_heads][head_dim] arrays.  A bit copy used by tests to
 * check the paging arithmetic the attention kernels share. */
mw_status mw_kv_pool_gather(const mw_kv_pool *pool, const int32_t *d_block_table,
                            int32_t n_tokens, void *d_k_out, void *d_v_out, mw_stream stream);

/* ------------------------------------------------------------------------
 * CU partition (Sec. 3.2.1: bind each phase's stream to its own compute
 * units; Sec. 5: hipExtStreamCreateWithCUMask on AMD GPUs).
 * MI355X has 8 XCDs of 32 CUs and dispatches workgroups round-robin over the
 * XCDs, so each partition takes the same number of CUs on every XCD: CU
 * counts must be multiples of 8, at least 8 each, and sum to at most the
 * device's CU count.  The masks are 32-bit words, bit i of word w naming
 * CU (32*w + i) in the runtime's CU numbering.
 * ---------------------------------------------------------------------- */
typedef struct mw_partition mw_partition;
/* Creates two streams on `device`: prefill on prefill_cus CUs and decode on
 * decode_cus disjoint CUs. */
mw_status mw_partition_create(int32_t device, int32_t prefill_cus, int32_t decode_cus,
                              mw_partition **out);
/* Same, from explicit masks of n_words 32-bit words each (must be disjoint
 * and non-empty). */
mw_status mw_partition_create_masks(int32_t device, const uint32_t *prefill_mask,
                                    const uint32_t *decode_mask, int32_t n_words,
                                    mw_partition **out);
mw_status mw_partition_streams(const mw_partition *part, mw_stream *prefill,
                               mw_stream *decode);
/* Copies the masks out (n_words = 8 words each, unused words zero). */
mw_status mw_partition_masks(const mw_partition *part, uint32_t *prefill_mask,
                             uint32_t *decode_mask);
/* Synchronises both streams, then destroys them. */
mw_status mw_partition_destroy(mw_partition *part);

/* Launches n_blocks one-wave workgroups on `stream` that each record the
 * hardware ids of the CU they run on and a start/end timestamp:
 * d_out[4*b + 0] = XCC id, [+1] = HW_ID register (CU, SIMD, shader array,
 * shader engine fields), [+2] = start and [+3] = end of a spin of spin_cycles
 * shader clocks (low 32 bits of the 100 MHz real-time counter).  `timing`
 * may be NULL; given one, it records the launch as one kernel. */
mw_status mw_cu_probe(int32_t n_blocks, int32_t spin_cycles, uint32_t *d_out,
                      mw_stream stream, mw_timing *timing);

/* Measured HBM read ceiling: reads `bytes` (a multiple of 16, 16-byte aligned)
 * from d_src once with n_blocks 256-thread work-groups on `stream` (so on that
 * stream's CUs) and writes one word per work-group to d_sink[n_blocks].  Used
 * to report attention bandwidth against what the same CUs can stream.
 * `timing` may be NULL. */
mw_status mw_stream_read(const void *d_src, size_t bytes, uint32_t *d_sink, int32_t n_blocks,
                         mw_stream stream, mw_timing *timing);

/* Measurement helpers (not part of the attention path).
 * mw_cache_flush: reads d_buf past its first 16 KiB on `stream` (bytes a
 *     multiple of 16 and above 16 KiB, 16-byte aligned) and writes one word
 *     per work-group (2048) into its first 8 KiB; with bytes >= 512 MiB it
 *     evicts the L2 caches of the stream's XCDs and the 256 MiB Infinity
 *     Cache, leaving clean lines only, so the next timed call starts cold.
 * mw_mfma_peak: n_blocks 256-thread work-groups each issuing `iters` rounds of
 *     four bf16 32x32x16 MFMAs per wave from registers, on `stream`; *flop
 *     (may be NULL) receives the launch's floating-point operations and
 *     d_sink[n_blocks] one folded value per work-group.  Timed with `timing`
 *     (may be NULL), it measures the matrix-core ceiling of the stream's CUs.
 * mw_trace_mark: launches an empty kernel (k_trace_mark) of `id` one-wave
 *     work-groups (1 <= id <= 65536), so that a kernel trace can find marked
 *     points of a program by that kernel's grid size. */
mw_status mw_cache_flush(void *d_buf, size_t bytes, mw_stream stream);
mw_status mw_mfma_peak(int32_t n_blocks, int32_t iters, float *d_sink, mw_stream stream, mw_timing *timing,
                       double *flop);
mw_status mw_trace_mark(int32_t id, mw_stream stream);

/* ------------------------------------------------------------------------
 * Per-call timing.  A call given a timing handle records a start event, one
 * event after each kernel it launches, and (implicitly) a stop event = the
 * last one, all on its stream.
 * ---------------------------------------------------------------------- */
mw_status mw_timing_create(mw_timing **out);
mw_status mw_timing_destroy(mw_timing *t);
/* Records only a start event on `stream` (a reference point for offsets). */
mw_status mw_timing_mark(mw_timing *t, mw_stream stream);
/* Waits for the stop event.  gpu_ms = stop - start; host_launch_ms = host
 * wall time the recording call spent enqueueing.  Either output may be NULL. */
mw_status mw_timing_elapsed(mw_timing *t, float *gpu_ms, float *host_launch_ms);
/* Number of kernels recorded and the GPU time of kernel k (event k to k+1). */
mw_status mw_timing_kernels(mw_timing *t, int32_t *n_kernels);
mw_status mw_timing_kernel_ms(mw_timing *t, int32_t k, float *ms);
/* Start and stop of t relative to ref's start event, in ms. */
mw_status mw_timing_offsets(mw_timing *t, mw_timing *ref, float *start_ms, float *stop_ms);

/* ------------------------------------------------------------------------
 * Attention.  For output row i of a sequence with nvis visible keys and query
 * head h (kv = h / (Hq/Hkv)):
 *     O[i][h] = softmax_j(scale * Q[i][h] . K[j][kv]) V[j][kv],  j < nvis
 * Prefill with a cached prefix (Sec. 3.3, Table "tab:theory_cost": n new
 * tokens against L = r + n keys; Sec. 1: a chunk reads the KV of every
 * earlier chunk): row i of a sequence with prefix r sees keys 0 .. r+i
 * (nvis = r + i + 1).  Decode (same table: r + 1 keys): the sequence's own
 * new K/V is already in the pool at position L-1, and its query sees keys
 * 0 .. L-1 (nvis = L).  Every K/V row is read through the block table.
 * ---------------------------------------------------------------------- */
typedef struct {
    int32_t num_q_heads;  /* multiple of num_kv_heads                      */
    int32_t num_kv_heads; /* must equal the pool's                         */
    int32_t head_dim;     /* must be 128                                   */
    float scale;          /* softmax scale, usually 1/sqrt(head_dim)       */
} mw_attn_shape;

/* Causal prefill for `batch` sequences (varlen).
 *   h_new_lens, h_prefix_lens host [batch]: n_b >= 0, r_b >= 0, with
 *       r_b + n_b <= bt_stride * page_size
 *   d_qo_indptr   device [batch+1]: rows of sequence b are
 *       [d_qo_indptr[b], d_qo_indptr[b+1]) of d_q / d_out
 *   d_prefix_lens device [batch]
 *   d_block_table device [batch][bt_stride]; must map every position
 *       < r_b + n_b (the new tokens' K/V are written before this call)
 *   d_q, d_out    device [sum n][num_q_heads][head_dim] bf16, 16-B aligned
 * One kernel launch; `timing` may be NULL. */
mw_status mw_prefill_attn(const mw_kv_pool *pool, const mw_attn_shape *shape, int32_t batch,
                          const int32_t *h_new_lens, const int32_t *h_prefix_lens,
                          const int32_t *d_qo_indptr, const int32_t *d_prefix_lens,
                          const int32_t *d_block_table, int32_t bt_stride, const void *d_q,
                          void *d_out, mw_stream stream, mw_timing *timing);

/* Prefill with a key-range split for grids too small to fill the stream's
 * CUs (the launches that run 32-position query blocks, two work-groups per
 * CU: a lone prefill on the whole device, a tensor-parallel head shard on a
 * partition).  There the longest causal block (its keys 0 .. r + i) sets the
 * call's time; the split cuts each block's key range into up to 8 equal
 * pieces so that the pieces fill about three rounds of the stream's
 * work-group slots, each piece computes the partial softmax state (reference
 * maximum m, row sum l, unnormalised output) of its keys into the workspace,
 * and a second kernel merges the pieces of every split block with the
 * log-sum-exp identity (the decode combine's merge; Table "tab:theory_cost"
 * fixes every row's key set, so the merged result is the same attention).
 * Without a split to make (a grid that fills the CUs, or blocks of at most
 * 4 key tiles) this is mw_prefill_attn: one launch, workspace unused.  With
 * one, two launches (split, merge), recorded as two kernels in `timing`.
 * The split depends on the lengths and on the stream's CU count, never on
 * page ids; rounding may differ from mw_prefill_attn in the last bits.
 *
 * Workspace bytes a call with these lengths may need on a stream of
 * num_cus CUs (0: the most any stream can need):
 *     pieces x sum(n) x num_q_heads x (128 x 4 + 8) */
mw_status mw_prefill_workspace_size(const mw_attn_shape *shape, int32_t batch, const int32_t *h_new_lens,
                                    const int32_t *h_prefix_lens, int32_t num_cus, size_t *bytes);
/* Arguments as mw_prefill_attn, plus d_workspace (device, 16-B aligned,
 * caller-owned, contents need not be initialised) of workspace_bytes.
 * MW_ERR_INVALID_ARG if the split this call makes needs more workspace than
 * given (the size call with this stream's CU count, or with 0, suffices). */
mw_status mw_prefill_attn_ws(const mw_kv_pool *pool, const mw_attn_shape *shape, int32_t batch,
                             const int32_t *h_new_lens, const int32_t *h_prefix_lens,
                             const int32_t *d_qo_indptr, const int32_t *d_prefix_lens,
                             const int32_t *d_block_table, int32_t bt_stride, const void *d_q, void *d_out,
                             void *d_workspace, size_t workspace_bytes, mw_stream stream, mw_timing *timing);

/* Decode streams each (sequence, kv head) segment of the K/V pages split into
 * pieces whose partial results are merged with the log-sum-exp combine (the
 * flash-decoding split of Sec. 2.2's memory-bound decode).  chunk_pages
 * chooses the split:
 *   0  (default) balanced: the segments laid end to end are cut into equal
 *      ranges of pages, two per CU of the stream the call runs on (at most
 *      512, at least 16 pages each); a range may cross segment boundaries and
 *      every CU streams the same number of bytes (when every sequence is
 *      long enough for two ranges or more, segments are padded to a multiple
 *      of the range instead, so that ranges do not straddle segments, if that
 *      keeps 90% of the work-groups).  The split depends on the lengths and
 *      on the stream's CU count.  One kernel: the work-group
 *      that finds every piece of a segment done (per-piece flags in the
 *      workspace, tagged per call, so the workspace needs no initialisation)
 *      merges that segment.
 *   -1 fixed chunks chosen from the lengths: the largest of 128, 64 and 32
 *      pages that still gives at least 1024 (chunk, kv head) work units.
 *   8..256, a multiple of 8: fixed chunks of that many pages; a second
 *      kernel merges the chunks.
 * No split ever depends on page ids (renumbering pages changes no result).
 * Pass the same chunk_pages (and lengths) to both calls; the size for 0
 * covers both splits that chunk_pages 0 can select (see mw_fused_attn).
 * Workspace bytes for a call with these lengths: */
mw_status mw_decode_workspace_size(const mw_attn_shape *shape, int32_t batch,
                                   const int32_t *h_seq_lens, int32_t chunk_pages,
                                   size_t *bytes);
/*   h_seq_lens host [batch], d_seq_lens device [batch]: L_b >= 1,
 *       L_b <= bt_stride * page_size
 *   d_block_table device [batch][bt_stride]
 *   d_q, d_out device [batch][num_q_heads][head_dim] bf16
 *   d_workspace device, >= mw_decode_workspace_size bytes, 16-B aligned;
 *       two calls that run at the same time need two workspaces
 * One kernel launch with the balanced split, two (split, combine) with fixed
 * chunks; `timing` may be NULL. */
mw_status mw_decode_attn(const mw_kv_pool *pool, const mw_attn_shape *shape, int32_t batch,
                         const int32_t *h_seq_lens, const int32_t *d_seq_lens,
                         const int32_t *d_block_table, int32_t bt_stride, const void *d_q,
                         void *d_out, void *d_workspace, size_t workspace_bytes,
                         int32_t chunk_pages, mw_stream stream, mw_timing *timing);

/* Decode attention that allocates nothing, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): mw_decode_attn with the same arguments, checks and
 * results (the same kernels and split), except that its workspace is a
 * library-owned static device array of 16 MiB per device, held until the
 * process ends, instead of d_workspace.  The call makes no hipMalloc, hipFree
 * or other allocating call; its first call on a device looks up that device's
 * array.  A call whose split needs more than 16 MiB of workspace (see
 * mw_decode_workspace_size) fails with MW_ERR_UNSUPPORTED before launching
 * anything.  Nothing in the array needs clearing between calls: a call reads
 * only what it wrote (the merge's done flags count only with the call's own
 * tag).  Every call on a device shares its array, so calls
 * that may overlap in time on one device (two streams, two threads) race:
 * order them on one stream or use mw_decode_attn.  No timing handle. */
mw_status mw_decode_attn_noalloc(const mw_kv_pool *pool, const mw_attn_shape *shape, int32_t batch,
                                 const int32_t *h_seq_lens, const int32_t *d_seq_lens,
                                 const int32_t *d_block_table, int32_t bt_stride, const void *d_q,
                                 void *d_out, int32_t chunk_pages, mw_stream stream);

/* ------------------------------------------------------------------------ *
 * Contention-tolerant estimator (paper Sec. 3.3) and the prefill-layer count
 * of the dispatcher (Sec. 3.4).  Host-side only: these calls touch no GPU.
 * ------------------------------------------------------------------------ */

/* Solo-run predictor (Sec. 3.3, "Solo-run predictor", Eqs. (1) and (2)):
 * per-call latency models fitted to measured solo runs, one model per phase
 * and per partition size (number of CUs the phase runs on):
 *     T_prefill = th1 * sum_i n_i^2 + th2 * sum_i n_i r_i + th3 * sum_i n_i + th4
 *     T_decode  = th1 * sum_i r_i + th2 * bs + th3
 * with n_i the new and r_i the reused (cached) tokens of sequence i; a decode
 * sequence of context length L has r = L - 1 (its own token is the new one).
 * The fit minimises the squared relative error (each sample's equation is
 * divided by its measured time), which is what the paper's accuracy figure
 * (maximum relative deviation) measures.  Times are in milliseconds.
 *
 *   mw_predictor_add_*: record one measured call.  Lengths are host arrays of
 *       `batch` entries (n >= 1, r >= 0; L >= 1); ms > 0 and finite.
 *   mw_predictor_fit: fits every (phase, cus) with at least as many samples
 *       as coefficients; MW_ERR_NOT_READY if none has.
 *   mw_predictor_*_ms: the model's prediction; MW_ERR_NOT_READY if no model
 *       was fitted for that phase and partition size.
 *   mw_predictor_coefficients: th1..th4 (prefill) or th1..th3 (decode, th[3]
 *       set to 0) of a fitted model.  phase: 0 = prefill (its 8-wave path
 *       once a launch shape is set), 1 = decode, 2 = prefill on the 4-wave
 *       path (launch shape set).
 *
 *   mw_predictor_set_launch_shape: tells the predictor the attention shape
 *       of the calls it models (query and kv heads; num_q_heads a multiple of
 *       num_kv_heads), before any prefill sample is added (else
 *       MW_ERR_INVALID_ARG).  A single attention call, unlike the paper's
 *       whole-model iterations, keeps the steps of its launch: rounds of
 *       work-groups over the partition's CUs, and calls whose few work-groups
 *       run at once, bound by the longest.  With the shape, each prefill
 *       call's launch on `cus` CUs is planned as mw_prefill_attn_ws plans it
 *       (key-range split included) and simulated: the work-groups in dispatch
 *       order, each to a CU slot that frees within 5% of the mean
 *       work-group's work of the earliest one, preferring the CU that holds
 *       the fewest work-groups so far (work-groups a tile or two apart finish
 *       together), a work-group's work its key tiles.  The n^2, n r and n terms of Eq. (1) are multiplied by the
 *       load-imbalance factor (the latest CU's time over the time of the same
 *       work spread evenly), and the kernel path (8-wave or 4-wave blocks)
 *       selects one of two models per partition size, fitted separately, as
 *       the paper keeps separate models for separate kernels.  Predicting
 *       with a path whose model is not fitted uses the other path's model;
 *       mw_predictor_fit leaves a 4-wave-path model whose samples do not
 *       determine it unfitted instead of failing.
 *       Decode keeps Eq. (2) as is. */
typedef struct mw_predictor mw_predictor;
mw_status mw_predictor_create(mw_predictor **out);
mw_status mw_predictor_destroy(mw_predictor *p);
mw_status mw_predictor_set_launch_shape(mw_predictor *p, int32_t num_q_heads, int32_t num_kv_heads);
mw_status mw_predictor_add_prefill(mw_predictor *p, int32_t cus, int32_t batch, const int32_t *new_lens,
                                   const int32_t *prefix_lens, double ms);
mw_status mw_predictor_add_decode(mw_predictor *p, int32_t cus, int32_t batch, const int32_t *seq_lens,
                                  double ms);
mw_status mw_predictor_fit(mw_predictor *p);
mw_status mw_predictor_prefill_ms(const mw_predictor *p, int32_t cus, int32_t batch, const int32_t *new_lens,
                                  const int32_t *prefix_lens, double *ms);
mw_status mw_predictor_decode_ms(const mw_predictor *p, int32_t cus, int32_t batch, const int32_t *seq_lens,
                                 double *ms);
mw_status mw_predictor_coefficients(const mw_predictor *p, int32_t phase, int32_t cus, double theta[4]);

/* Contention guard (Sec. 3.3, "Contention guard"): the maximum decode
 * slowdown (multiplexed / solo latency) seen in each cell of a grid over five
 * variables: prefill new tokens, prefill reused tokens, decode batch size,
 * decode reused tokens in total, and the prefill partition size.  Token
 * counts fall into powers-of-4 cells (x in (4^(k-1), 4^k] is cell k; 0 and 1
 * are cell 0), batch sizes into powers-of-2 cells, the partition size is
 * matched exactly.  Samples raise a cell's maximum, so the guard can keep
 * learning from run-time measurements.
 *   mw_guard_add: slowdown > 0 and finite; counts >= 0, batch >= 1, cus >= 1.
 *   mw_guard_lookup: the cell's maximum; for a cell without samples the
 *       maximum over all cells of the same partition size, then over all
 *       cells; 1.0 for an empty guard.
 * Worst-case decode latency = predicted solo latency x guard slowdown. */
typedef struct {
    int64_t prefill_new, prefill_reused, decode_batch, decode_reused;
    int32_t prefill_cus;
} mw_guard_key;
typedef struct mw_guard mw_guard;
mw_status mw_guard_create(mw_guard **out);
mw_status mw_guard_destroy(mw_guard *g);
mw_status mw_guard_add(mw_guard *g, const mw_guard_key *key, double slowdown);
mw_status mw_guard_lookup(const mw_guard *g, const mw_guard_key *key, double *slowdown);

/* Number of prefill layers to launch next to one decode iteration (Sec. 3.4):
 * N_PL = ceil(T_d * N_T / T_P) with T_d the estimated decode latency, T_P the
 * estimated latency of the whole prefill and N_T the model's layer count;
 * the result is clamped to [1, N_T].  Times > 0 and finite, n_layers >= 1. */
mw_status mw_prefill_layers(double t_decode_ms, double t_prefill_ms, int32_t n_layers, int32_t *n_pl);

/* ------------------------------------------------------------------------ *
 * Bubble-less multiplex engine (paper Sec. 3.2, "Bubble-less Multiplex
 * Engine"): a group of CU partitions created once, and a host loop that
 * feeds decode iterations and prefill layers to their streams.
 *
 * The paper's engine splits prefill into layers, launches N_PL layers at a
 * time next to each decode iteration, polls events instead of blocking
 * ("query-based synchronization") and moves the remaining prefill layers to
 * a new partition when decode ends.  Here a decode iteration is
 * `decode_layers` decode attention calls and the prefill job is
 * `prefill_layers` prefill attention calls (one per transformer layer, made
 * with the same arguments each time: the attention hot path of the layers,
 * not the rest of the model).
 *
 * mw_engine_create: one partition per entry of prefill_cus[0..n) (prefill on
 *     that many CUs, decode on the device's other CUs; multiples of 8), plus
 *     a stream on the whole device; 1 <= n <= 16.  The device memory the
 *     group takes (free memory before minus after) and the creation time are
 *     reported by mw_engine_memory.
 * mw_engine_streams: the prefill and decode streams of partition `config`
 *     (config = -1: the whole-device stream in both).
 * mw_engine_run: one multiplexed run on partition plan->config; blocks until
 *     every call it launched has completed, then fills `stats`.  Device
 *     buffers are the caller's, as for mw_decode_attn / mw_prefill_attn;
 *     lengths arrays are host copies read at launch time.
 *   policy MW_ENGINE_BLOCKING: launch decode iteration 0, then the whole
 *     prefill job, and wait (blocking) for each decode iteration before
 *     launching the next; the prefill keeps its partition to the end.
 *   policy MW_ENGINE_POLLED: launch decode iteration 0 and N_PL =
 *     plan->layers_per_launch prefill layers; then poll: a finished decode
 *     iteration is followed at once by the next, and prefill layers are
 *     topped up N_PL at a time whenever fewer than N_PL are queued; with
 *     plan->switch_on_decode_end the layers launched after the last decode
 *     iteration ends go to the whole-device stream (ordered after the
 *     earlier layers by a cross-stream event wait).
 *   plan->decode_graph = 1: a decode iteration is launched as one HIP graph
 *     (paper Sec. 3.2: graphs for the decode phase only, one per batch size
 *     and partition).  The engine captures it on the partition's decode
 *     stream at the first run with these decode arguments, lengths, layer
 *     count and partition, keeps it until mw_engine_destroy, and replays it
 *     on later runs; the capture is outside the timed run.  The graph holds
 *     the device pointers and lengths it was captured with: a caller that
 *     changes the buffers' contents gets them read again, one that changes a
 *     pointer or a length gets a new graph.  Stats then time each iteration
 *     as one span.
 * Stats (device times from HIP events around every call, in ms from the
 * first launch): each stream's busy time (sum of its calls) and bubble ratio
 * (1 - busy / its first-start-to-last-end window), their mean, the longest
 * gap between consecutive decode iterations, the prefill job's end, and at a
 * partition switch the gap on the prefill timeline and the host time of the
 * switch itself (the cross-stream wait and the change of stream, not the
 * launches that follow).  Each event pair adds a marker packet per call, so
 * the bubbles include that marker time (a few microseconds per call).
 * Errors: MW_ERR_INVALID_ARG for a NULL pointer, a config outside [0, n), a
 * count below 1 or an unknown policy (nothing launched); the argument
 * checks of mw_decode_attn / mw_prefill_attn on the first launch; MW_ERR_HIP
 * for a HIP failure, returned after every launched call has completed.  The
 * engine owns its streams and events only; one run at a time per engine. */
typedef struct mw_engine mw_engine;
enum { MW_ENGINE_BLOCKING = 0, MW_ENGINE_POLLED = 1 };
typedef struct {
    const mw_kv_pool *pool;
    mw_attn_shape shape;
    int32_t batch;
    const int32_t *h_seq_lens, *d_seq_lens, *d_block_table;
    int32_t bt_stride;
    const void *d_q;
    void *d_out, *d_workspace;
    size_t workspace_bytes;
    int32_t chunk_pages;
} mw_decode_args;
typedef struct {
    const mw_kv_pool *pool;
    mw_attn_shape shape;
    int32_t batch;
    const int32_t *h_new_lens, *h_prefix_lens, *d_qo_indptr, *d_prefix_lens, *d_block_table;
    int32_t bt_stride;
    const void *d_q;
    void *d_out;
    void *d_workspace;      /* NULL: the plain call (mw_prefill_attn); else the */
    size_t workspace_bytes; /* key-range split's workspace (mw_prefill_attn_ws) */
} mw_prefill_args;
typedef struct {
    int32_t config;             /* partition index, 0 <= config < n */
    int32_t decode_iters;       /* >= 1 */
    int32_t decode_layers;      /* decode calls per iteration, >= 1 */
    int32_t prefill_layers;     /* prefill calls of the job, >= 1 */
    int32_t layers_per_launch;  /* N_PL, >= 1 (polled policy) */
    int32_t policy;             /* MW_ENGINE_BLOCKING or MW_ENGINE_POLLED */
    int32_t switch_on_decode_end;
    int32_t decode_graph;       /* 1: each decode iteration is one graph launch */
} mw_engine_plan;
typedef struct {
    double wall_ms;                       /* first launch to last completion */
    double decode_busy_ms, prefill_busy_ms;
    double decode_bubble, prefill_bubble, bubble_ratio;
    double decode_gap_ms_max;             /* longest idle gap between decode iterations */
    double decode_iter_ms_mean;           /* decode iteration, first call start to last call end */
    double prefill_end_ms;                /* completion of the last prefill layer */
    double switch_gap_ms;                 /* prefill timeline gap at the switch; -1 if none */
    double switch_host_us;                /* host time of the switch; -1 if none */
    double host_launch_ms;                /* host time spent launching */
    double decode_launch_us_mean;         /* host time to launch one decode iteration */
    int32_t prefill_batches;              /* launch decisions that launched prefill layers */
    int32_t switched_layers;              /* prefill layers run on the whole device */
} mw_engine_stats;
/* One launch covering a prefill call and a decode call on the same pool: the
 * fused comparator (paper Sec. 4.1: the chunked-prefill baseline runs prefill
 * and decode attention in one kernel on the whole GPU).  Each work-group of
 * the fused kernel is either one prefill work-group or two decode work
 * units; the two kinds are interleaved in dispatch order in proportion to
 * their counts, then the decode combine kernel runs.  Arguments, layouts and
 * results are those of mw_prefill_attn (pre) and mw_decode_attn (dec) with
 * the same checks; both must name the same pool, and the prefill outputs must
 * not overlap the decode outputs or workspace.  The decode work units are
 * fixed chunks (dec->chunk_pages 0 is taken as -1: the balanced split's
 * units differ in their number of work-group barriers, which the two halves
 * of a fused work-group cannot).  Outputs are bit-identical to the two
 * separate calls with the same chunks.  timing records 2 kernels (fused,
 * combine). */
mw_status mw_fused_attn(const mw_prefill_args *pre, const mw_decode_args *dec, mw_stream stream,
                        mw_timing *timing);

mw_status mw_engine_create(int32_t device, const int32_t *prefill_cus, int32_t n, mw_engine **out);
mw_status mw_engine_destroy(mw_engine *eng);
mw_status mw_engine_streams(const mw_engine *eng, int32_t config, mw_stream *prefill, mw_stream *decode);
mw_status mw_engine_memory(const mw_engine *eng, int64_t *device_bytes, double *create_ms);
mw_status mw_engine_run(mw_engine *eng, const mw_decode_args *dec, const mw_prefill_args *pre,
                        const mw_engine_plan *plan, mw_engine_stats *stats);

/* Captured decode graphs of `eng`: their count, the device memory their
 * instantiation and upload took (free memory before minus after, summed)
 * and the host time of capture + instantiation + upload.  Outputs may be
 * NULL. */
mw_status mw_engine_graphs(const mw_engine *eng, int32_t *n_graphs, int64_t *device_bytes, double *capture_ms);

/* Per-call timeline of the last mw_engine_run on `eng`: phase 0 = decode
 * calls, 1 = prefill calls, in launch order.  Writes min(n_calls, capacity)
 * rows of three doubles (start ms, end ms, 1 if the call ran on the whole
 * device after a switch, else 0), times relative to the run's reference
 * event, to the host array `out`; *n_calls receives the number of calls.
 * capacity 0 only queries the count. */
mw_status mw_engine_timeline(const mw_engine *eng, int32_t phase, double *out, int32_t capacity,
                             int32_t *n_calls);

#ifdef __cplusplus
}
#endif

#endif /* MW_H */
