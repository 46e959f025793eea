/*
 * art_oracle.h -- CPU reference ("oracle") for ART decode attention.
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the slow, plain, fp64 statement
 * of what the GPU path must compute; only the test-suite, the smoke check and
 * the benchmark's CPU-baseline leg may load it.  It shares no code, header,
 * table or helper with the HIP library.
 *
 * What it computes (per (sequence b, KV head kvh) group, query heads
 * h = kvh*g .. kvh*g+g-1, g = num_q_heads / num_kv_heads):
 *   - the traversal list of KV blocks: dense recency-first (Sec. 3.4, full KV
 *     cache), dense forward, or a caller-supplied block list (Sec. 3.4,
 *     importance-first through an index mapping);
 *   - for t = 1..T the block-streaming softmax of Sec. 3.1 in the normalised
 *     form of Appendix A: o(t) = (A(t-1) o(t-1) + l(t) u(t)) / A(t);
 *   - the stability metrics of Eq. (2) on the probe x(t) = P o(t):
 *     d_scale = ||x(t) - x(t-1)||_2 and d_direction = 1 - cos(x(t), x(t-1))
 *     with o(0) = 0 (Algorithm 1);
 *   - the patience counter of Eq. (3) and the break of Algorithm 1;
 *   - out = o(t*), lse = ln A(t*), stop_block = t*.
 * Readings where the paper is silent are listed in the .c file header.
 */
#ifndef ART_ORACLE_H
#define ART_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t batch;
    int32_t num_q_heads;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t block_size;           /* tokens per KV block (the unit of one step) */
    int32_t page_size;            /* tokens per cache page */
    int32_t num_pages;            /* pages in the pool */
    int32_t max_pages_per_seq;    /* row stride of page_table */
    int32_t max_blocks_per_list;  /* row stride of block_list */
    int32_t list_per_head;        /* 1: one list per (b, kvh); 0: one per b */
    int64_t k_stride_page, k_stride_head, k_stride_token;  /* elements */
    int64_t v_stride_page, v_stride_head, v_stride_token;
} artref_shape;

typedef struct {
    double scale;        /* softmax scale, the fp32 value the kernel gets, widened */
    double tau;          /* d_scale threshold (strict <) */
    double phi;          /* d_direction threshold (strict <) */
    int32_t patience;    /* p >= 1 */
    int32_t dense_order; /* 0: recency-first, 1: forward; ignored with a list */
    int32_t probe_stride; /* probe x = P o (Sec. 3.2, Appendix A): 1 = the whole
                             output (P = I); s > 1 (s divides head_dim) = the
                             coordinates 0, s, 2s, ... of o (m = head_dim / s) */
    int32_t scale_of_accumulator; /* 1: d_scale on the unnormalised accumulator
                             l(t) o(t), l(t) = sum of exp(s - running max), as
                             Algorithm 1 keeps it before its final normalisation
                             (R2 variant); 0: on o(t) */
    int32_t per_head_stop; /* 1: every query head has its own patience counter and
                             stop (R3 variant); the group reads blocks until all its
                             heads have stopped; 0: one stop per group */
} artref_opts;

enum {
    ARTREF_OK = 0,
    ARTREF_ERR_ARG = 1,
    ARTREF_ERR_INDEX = 5   /* block id out of range / duplicated, page id out of pool */
};

/*
 * q, k_cache, v_cache: bf16 bit patterns (host memory).
 * block_list / block_list_len: NULL for the dense traversal.
 * force_stop: NULL, or [batch][num_kv_heads] (with per_head_stop:
 *   [batch][num_q_heads], one value per query head); a value f >= 1 makes
 *   group (b, kvh) (or that query head) stop after step min(f, T)
 *   regardless of the criterion.
 * group_mask: NULL, or [batch][num_kv_heads]; groups with 0 are skipped
 *   (their outputs are left untouched).
 * out [batch][num_q_heads][head_dim], lse [batch][num_q_heads] (fp64),
 * stop_block [batch][num_kv_heads] (blocks the group consumed).
 * head_stop: NULL, or [batch][num_q_heads]: the stop of each query head (with
 *   per_head_stop; otherwise its group's stop).
 * trace: NULL, or [batch][num_kv_heads][trace_steps][g][2] holding
 *   (d_scale, d_direction) for steps 1..min(T, trace_steps) (NaN elsewhere).
 * num_threads <= 0: OpenMP default.
 * Returns ARTREF_OK, or an error code with *err_group = b*num_kv_heads+kvh.
 */
int artref_decode(const artref_shape* shape, const artref_opts* opts,
                  const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                  const int32_t* page_table, const int32_t* seq_lens,
                  const int32_t* block_list, const int32_t* block_list_len,
                  const int32_t* force_stop, const uint8_t* group_mask,
                  double* out, double* lse, int32_t* stop_block, int32_t* head_stop,
                  double* trace, int32_t trace_steps,
                  int32_t num_threads, int32_t* err_group);

/* number of OpenMP threads the library would use for num_threads <= 0 */
int artref_max_threads(void);

#ifdef __cplusplus
}
#endif
#endif
