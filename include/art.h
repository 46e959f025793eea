/*
 * art.h -- C ABI of the ART decode-attention library (libart.so, gfx950).
 *
 * ART (Attention Run-time Termination) computes single-query grouped-query
 * decode attention over a paged KV cache block by block with an online
 * softmax (Sec. 3.1, Eq. 1), and after every block tests whether the running
 * attention output has stabilised in magnitude and direction (Sec. 3.2,
 * Eq. 2).  Once the test has held for `patience` consecutive blocks (Eq. 3,
 * Algorithm 1) it stops reading the remaining KV blocks.  The block order is
 * recency-first or forward over the whole cache, or a caller-supplied list of
 * block ids (importance-first traversal through an index mapping, Sec. 3.4).
 *
 * Definition computed (per sequence b and KV head kvh, query heads
 * h = kvh*g .. kvh*g+g-1 with g = num_q_heads / num_kv_heads):
 *   traversal blocks B_1..B_T; o(0) = 0; for t = 1..T
 *     o(t) = softmax-weighted mean of V over the tokens of B_1..B_t
 *            (Appendix A's normalised recurrence),
 *     d_scale(t) = ||o(t) - o(t-1)||_2, d_direction(t) = 1 - cos(o(t), o(t-1))
 *     per query head; the step is stable iff every head of the group has
 *     d_scale < tau and d_direction < phi (a zero vector makes the step
 *     unstable, so step 1 never is);
 *     c(t) = stable ? c(t-1) + 1 : 0; stop at the first t with c(t) >= p.
 *   Outputs: out = o(t*), lse = ln(sum of exp(scale q.k)) over the consumed
 *   tokens, stop_block = t* (T when the test never fires, 0 when T = 0).
 *
 * Conventions
 *   - Every array pointer is DEVICE memory owned by the caller; the library
 *     allocates nothing per call.  Calls are asynchronous on `stream`.
 *   - Host-side checks return a status before anything is launched; a failed
 *     launch returns ART_ERR_HIP.  Nothing is thrown across the ABI.
 *   - Index arrays (page_table, block_list, seq_lens) are read on the device
 *     and clamped into range there, so malformed indices never make the
 *     kernel read outside the arrays described by the shape; the result for
 *     such input is unspecified.  art_validate_inputs() checks them exactly.
 *   - A workspace is caller-provided device memory of at least
 *     art_decode_workspace_bytes() bytes, filled with zeros once before its
 *     first use (art_workspace_init).  Each call leaves it ready for the next
 *     one.  One workspace serves one call at a time: calls that share it must
 *     be ordered (for example, issued on the same stream).
 *   - Results are deterministic: identical inputs, shape and options give
 *     bit-identical out, lse and stop_block whatever the scheduling.
 *   - The library is thread-safe; it keeps no mutable state except a
 *     process-wide call counter.
 */
#ifndef ART_H
#define ART_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ART_ABI_VERSION 8

typedef enum {
    ART_OK = 0,
    ART_ERR_INVALID_ARG = 1,        /* null pointer, negative size, bad enum, NaN threshold */
    ART_ERR_UNSUPPORTED = 2,        /* valid but not implemented (see art_decode_shape) */
    ART_ERR_WORKSPACE_TOO_SMALL = 3,
    ART_ERR_HIP = 4,                /* a HIP runtime call or launch failed */
    ART_ERR_BAD_INDEX = 5,          /* art_validate_inputs: an index is out of range or repeated */
    ART_ERR_DEVICE_TIMEOUT = 6      /* a kernel gave up waiting (reported by art_workspace_status) */
} art_status;

typedef enum { ART_ORDER_RECENT_FIRST = 0, ART_ORDER_FORWARD = 1 } art_order;
typedef enum { ART_OUT_F32 = 0, ART_OUT_BF16 = 1 } art_out_dtype;

/*
 * Problem shape.  Element strides are in elements (bf16); the head_dim
 * stride is 1.  Supported: head_dim == 128; g = num_q_heads / num_kv_heads in
 * {1, 2, 4, 8, 16}; block_size a multiple of 64 of at most 1024 tokens;
 * page_size a power of two >= 16; traversals (max_pages_per_seq * page_size
 * / block_size, and max_blocks_per_list) shorter than 2^19 blocks.  Anything
 * else returns ART_ERR_UNSUPPORTED.
 */
typedef struct {
    int32_t batch;
    int32_t num_q_heads;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t block_size;            /* tokens per KV block: the unit of one stability step */
    int32_t page_size;             /* tokens per cache page */
    int32_t num_pages;             /* pages in the K and V pools (page ids are < num_pages) */
    int32_t max_pages_per_seq;     /* row stride of page_table; seq_lens[b] <= max_pages_per_seq * page_size */
    int32_t max_blocks_per_list;   /* row stride of block_list (0 when no list is passed) */
    int32_t list_per_head;         /* 1: one list per (b, kvh); 0: one list per b shared by its KV heads */
    int64_t k_stride_page, k_stride_head, k_stride_token;
    int64_t v_stride_page, v_stride_head, v_stride_token;
} art_decode_shape;

/*
 * Options.  tau and phi are compared with a strict '<' (Algorithm 1):
 * tau <= 0 or phi <= 0 means the test never passes (no termination); +inf
 * removes that half of the test (the ablations of Table 3).  patience >= 1;
 * patience = 1 is "no patience"; INT32_MAX runs the detector without ever
 * stopping.  chunk_blocks = 0 lets the library pick the split of each
 * traversal into chunks from the shape alone (never from the data or the
 * thresholds: four leading chunks of 3 blocks, then chunks of up to 9);
 * 1..16 asks for that many blocks in every chunk (capped at what the
 * shared-memory budget holds for the shape).  The chunking changes
 * rounding only.
 *
 * probe_stride chooses the probe x(t) = P o(t) that the stability test of
 * Eq. (2) looks at (Sec. 3.2; P is the linear map of Appendix A): 0 or 1
 * tests the whole normalised output of every query head (P = I); s > 1,
 * a power of two dividing head_dim, tests only its coordinates 0, s, 2s,
 * ... (m =
 * head_dim / s values spread over the head dimension, a fixed stand-in for
 * the subsample Sec. 3.2 takes from the accumulator's register layout; the
 * paper's m = 32 is s = 4).  The output and lse are always the full ones.
 *
 * scale_of_accumulator = 1 takes d_scale on the unnormalised accumulator
 * X(t) = l(t) o(t) instead of o(t).  Here l(t) is the sum of exp(s - m(t))
 * over the consumed tokens, with m(t) the running maximum score.  X(t) is
 * what Algorithm 1 carries before its final normalisation, each step in its
 * own reference.  The other reading of Algorithm 1; d_direction is the same
 * under both.
 */
typedef struct {
    float softmax_scale;           /* usually 1/sqrt(head_dim) (Eq. 1) */
    float tau;                     /* d_scale threshold */
    float phi;                     /* d_direction = 1 - cos threshold */
    int32_t patience;
    int32_t dense_order;           /* art_order; ignored when block_list != NULL */
    int32_t out_dtype;             /* art_out_dtype */
    int32_t chunk_blocks;          /* 0 = automatic */
    int32_t probe_stride;          /* 0 or 1 = whole output; s > 1 = every s-th coordinate */
    int32_t scale_of_accumulator;  /* 0: d_scale on o(t); 1: on the accumulator l(t) o(t) */
    int32_t no_detector;           /* 1: no stability test at all (tau, phi, patience and
                                      the probe options are ignored): full attention over
                                      the traversal, stop_block = T; the baseline that
                                      shows what the test itself costs */
    int32_t max_wait_polls;        /* 0 = default (2^22 polls of about a microsecond each);
                                      n > 0: a wait on another workgroup's chunk gives up
                                      after n polls (a watchdog; see art_workspace_status) */
    int32_t per_head_stop;         /* 0: one stop per (sequence, KV head): a step is stable
                                      only if it is for every query head of the group;
                                      1: every query head keeps its own patience counter
                                      (Eq. 3) and stops on its own; its out and lse are
                                      those at its own stop, and stop_block is then
                                      [batch][num_q_heads]: each head's stop (T if it never
                                      stops).  A group reads blocks until its last head
                                      has stopped.  Needs a larger workspace
                                      (art_decode_workspace_bytes) */
    int32_t max_ahead_chunks;      /* 0 = unbounded; n > 0 bounds the reads past a stop:
                                      chunk k of a traversal is not loaded before chunk
                                      k - n of it has been through the stability test
                                      (or a stop before chunk k is known), so at most n
                                      chunks are read past the one that decides the stop.
                                      It changes which blocks are read, never the
                                      results (the outputs are bit for bit those of the
                                      unbounded call); it can idle workgroups, so the
                                      launch may take longer */
} art_decode_opts;

/* Version of this ABI (ART_ABI_VERSION). */
int32_t art_abi_version(void);

/* Human-readable name of a status code (static string). */
const char* art_status_str(int32_t status);

/*
 * Workspace bytes the call with this shape and these options needs (a
 * function of the shape only).  Returns 0 and sets *status on invalid input.
 */
size_t art_decode_workspace_bytes(const art_decode_shape* shape,
                                  const art_decode_opts* opts, int32_t* status);

/* Zero-fill `bytes` of workspace on `stream` (asynchronous; a plain kernel,
 * so it may be captured in a HIP graph). */
art_status art_workspace_init(void* workspace, size_t bytes, hipStream_t stream);

/*
 * ART decode attention (Algorithm 1 with the readings above).
 *   q            bf16 [batch][num_q_heads][head_dim], contiguous.
 *   k_cache      bf16 pool; token `s` of page `p` of KV head `h` starts at
 *   v_cache        k_cache + p*k_stride_page + h*k_stride_head + s*k_stride_token.
 *   page_table   int32 [batch][max_pages_per_seq]: physical page of logical
 *                page i of sequence b (token j is in logical page j / page_size).
 *   seq_lens     int32 [batch], tokens in the cache per sequence (>= 0).
 *   block_list   NULL for the dense traversal (dense_order); otherwise int32
 *                [batch][list_per_head ? num_kv_heads : 1][max_blocks_per_list]
 *                logical block ids (block i holds tokens [i*block_size,
 *                min((i+1)*block_size, seq_len))) in traversal order; ids must
 *                be unique and < ceil(seq_len / block_size).
 *   block_list_len int32 [batch][list_per_head ? num_kv_heads : 1]; NULL iff
 *                block_list is NULL.  0 gives an empty traversal.
 *   out          [batch][num_q_heads][head_dim], fp32 or bf16 (out_dtype).
 *   lse          fp32 [batch][num_q_heads], natural log; -inf for T = 0.
 *   stop_block   int32 [batch][num_kv_heads]: blocks consumed t* (0..T);
 *                with per_head_stop, [batch][num_q_heads]: each head's stop.
 *   workspace    see art_decode_workspace_bytes / art_workspace_init.
 * Returns ART_OK once the work is enqueued.  Each call tags the workspace
 * with a fresh value of a host-side counter that is passed as a kernel
 * argument, so a call captured in a HIP graph must not be replayed: a
 * replay would reuse the captured tag.
 */
art_status art_decode_attention(const art_decode_shape* shape, const art_decode_opts* opts,
                                const void* q, const void* k_cache, const void* v_cache,
                                const int32_t* page_table, const int32_t* seq_lens,
                                const int32_t* block_list, const int32_t* block_list_len,
                                void* out, float* lse, int32_t* stop_block,
                                void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/*
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * decode call (same kernels, same plan, bit-identical results) with the
 * library's own scratch in place of the caller's workspace: a static device
 * array of ART_STATIC_SCRATCH_BYTES per GPU, held from the library's first
 * use on that GPU until the process ends.  The call allocates nothing; on
 * its first use on a device (the current device) it takes the array's
 * address and zero-fills it on `stream`.
 *   - Arguments as for art_decode_attention, without the workspace.
 *   - A shape whose art_decode_workspace_bytes() exceeds
 *     ART_STATIC_SCRATCH_BYTES returns ART_ERR_WORKSPACE_TOO_SMALL before
 *     anything is launched.
 *   - Every call on one GPU shares that GPU's array: calls that overlap on a
 *     GPU (different streams, or host threads issuing concurrently) race.
 *     Order them, for example on one stream.
 *   - Each call tags what it leaves in the array with a fresh value of the
 *     call counter, so nothing needs clearing between calls (as for a
 *     workspace), and a captured call must not be replayed.
 *   - Bounded waits end the launch as in art_decode_attention; the error
 *     word lives in the array and is not reported by this call.
 */
#define ART_STATIC_SCRATCH_BYTES ((size_t)64 << 20)

art_status art_decode_attention_static(const art_decode_shape* shape, const art_decode_opts* opts,
                                       const void* q, const void* k_cache, const void* v_cache,
                                       const int32_t* page_table, const int32_t* seq_lens,
                                       const int32_t* block_list, const int32_t* block_list_len,
                                       void* out, float* lse, int32_t* stop_block,
                                       hipStream_t stream);

/*
 * Checked mode: synchronously copies the index arrays to the host and checks
 * seq_lens (0 <= L <= max_pages_per_seq * page_size), the page ids each
 * sequence uses (0 <= id < num_pages), and the block lists (ids in range,
 * unique, length <= max_blocks_per_list).  Returns ART_OK, an argument error,
 * or ART_ERR_BAD_INDEX with *bad_index set to the flat index of the first
 * offending element (into seq_lens, page_table, block_list or
 * block_list_len, in that order of checking; *bad_where = 0, 1, 2, 3).
 */
art_status art_validate_inputs(const art_decode_shape* shape, const art_decode_opts* opts,
                               const int32_t* page_table, const int32_t* seq_lens,
                               const int32_t* block_list, const int32_t* block_list_len,
                               hipStream_t stream, int64_t* bad_index, int32_t* bad_where);

/*
 * Synchronises `stream` and reports whether any call that used this workspace
 * since its initialisation gave up waiting on a predecessor chunk (a bounded
 * spin that ends the kernel instead of hanging it).  *device_status receives
 * ART_OK or ART_ERR_DEVICE_TIMEOUT.
 *
 * Every wait of the decode kernel is bounded (max_wait_polls).  The first
 * wave that gives up records the call in the workspace's error word; every
 * other wait of that call then ends within a few polls, so the launch
 * drains promptly.  The outputs of such a call are unspecified (some groups
 * may be left unwritten).  The error stays recorded until the workspace is
 * initialised again; later calls on the workspace run normally.
 */
art_status art_workspace_status(const void* workspace, size_t workspace_bytes,
                                hipStream_t stream, int32_t* device_status);

/*
 * Traversal lists (Sec. 3.4).  ART stops early only if the blocks that carry
 * the attention mass come first.  For a full cache the decode call itself
 * walks recency-first (dense_order).  For other KV policies it takes a
 * block list.  These calls build one on the device, in the decode call's
 * list layout (list_per_head = 1):
 *
 *   ART_LIST_IMPORTANCE  every block of each (sequence, KV head) gets a score.
 *       The first `sink_blocks` blocks, and the last block when keep_last = 1,
 *       are always kept.  Of the other blocks, the best `budget` minus (the
 *       kept count) are added.  The list holds the kept blocks in descending
 *       score order; equal scores put the smaller block id first.  Scores are
 *       doubles, each sum taken over dimensions 0..127 in order from exact
 *       products of the bf16 inputs:
 *         ART_SCORE_KEY_NORM:    max over the block's tokens of sum_d k_d^2.
 *         ART_SCORE_QUERY_BOUND: max over the group's query heads of
 *                                sum_d max(q_d * min_j k_jd, q_d * max_j k_jd),
 *                                which bounds q . k_j over the block from above.
 *       Keys and queries that hold a NaN give unspecified scores.
 *   ART_LIST_STREAMING  a cache of sink tokens plus a recent window
 *       (pattern-based policies).  Blocks 0 .. sink_blocks-1 come first, in
 *       increasing order, so that a stop never drops the sinks.  Then come the
 *       `budget` most recent other blocks, newest first.  No scores.
 *
 * Tokens at or beyond seq_len are not part of any block.  An empty sequence
 * gets an empty list.
 */
typedef enum { ART_LIST_IMPORTANCE = 0, ART_LIST_STREAMING = 1 } art_list_policy;
typedef enum { ART_SCORE_KEY_NORM = 0, ART_SCORE_QUERY_BOUND = 1 } art_score_kind;

typedef struct {
    int32_t policy;        /* art_list_policy */
    int32_t score_kind;    /* an art_score_kind; importance lists only */
    int32_t budget;        /* importance: blocks kept; streaming: recent blocks kept (>= 0) */
    int32_t sink_blocks;   /* leading blocks always kept (>= 0) */
    int32_t keep_last;     /* importance: 1 keeps the last (newest) block */
} art_list_opts;

/*
 * Workspace bytes art_build_block_list needs for the block scores when it
 * does not get a `block_scores` array: batch * num_kv_heads * max_blocks
 * doubles.  max_blocks = ceil(max_pages_per_seq * page_size / block_size)
 * must be at most 8192.  Shape fields used: batch, num_q_heads,
 * num_kv_heads, head_dim (128), block_size, page_size (a power of two),
 * num_pages, max_pages_per_seq, max_blocks_per_list (the row stride of the
 * output, which must hold the longest list the options allow), list_per_head
 * (must be 1) and the K strides (multiples of 8 elements).  Returns 0 and
 * sets *status on invalid input.
 */
size_t art_block_list_workspace_bytes(const art_decode_shape* shape, const art_list_opts* opts,
                                      int32_t* status);

/*
 * Build the lists on `stream` (asynchronous).
 *   q            bf16 [batch][num_q_heads][head_dim] (ART_SCORE_QUERY_BOUND only;
 *                may be NULL otherwise).
 *   k_cache, page_table, seq_lens  as for art_decode_attention.  k_cache and
 *                page_table may be NULL for streaming lists.
 *   block_list   int32 [batch][num_kv_heads][max_blocks_per_list], out.  Entries
 *                past a row's length are left as they were.
 *   block_list_len int32 [batch][num_kv_heads], out.
 *   block_scores NULL, or double [batch][num_kv_heads][max_blocks], out (the
 *                importance scores; entries of blocks past a sequence's end are
 *                left as they were).  When NULL, the workspace holds them.
 *   workspace    device memory of art_block_list_workspace_bytes() bytes, or
 *                none when block_scores is given or the list is streaming.
 * The outputs feed art_decode_attention directly (list_per_head = 1).
 */
art_status art_build_block_list(const art_decode_shape* shape, const art_list_opts* opts,
                                const void* q, const void* k_cache, const int32_t* page_table,
                                const int32_t* seq_lens, int32_t* block_list,
                                int32_t* block_list_len, double* block_scores,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* ART_H */
