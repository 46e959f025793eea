/*
 * art_list_oracle.h -- CPU reference for ART's traversal lists.
 *
 * TEST INFRASTRUCTURE ONLY: the plain fp64 statement of the lists the GPU
 * list producer must build (Sec. 3.4); only the test-suite may load it.  It
 * shares no code with the HIP library.  Readings are listed in the .c file.
 */
#ifndef ART_LIST_ORACLE_H
#define ART_LIST_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t batch, num_q_heads, num_kv_heads, head_dim;
    int32_t block_size, page_size, num_pages, max_pages_per_seq;
    int32_t max_blocks_per_list;   /* row stride of the output list */
    int64_t k_stride_page, k_stride_head, k_stride_token;   /* elements */
} artref_list_shape;

enum { ARTREF_LIST_IMPORTANCE = 0, ARTREF_LIST_STREAMING = 1 };
enum { ARTREF_SCORE_KEY_NORM = 0, ARTREF_SCORE_QUERY_BOUND = 1 };

typedef struct {
    int32_t policy;       /* ARTREF_LIST_* */
    int32_t score_kind;   /* ARTREF_SCORE_* (importance lists) */
    int32_t budget;       /* importance: blocks selected; streaming: recent blocks kept */
    int32_t sink_blocks;  /* leading blocks always kept */
    int32_t keep_last;    /* importance: the last block is always kept */
} artref_list_opts;

enum { ARTREF_LIST_OK = 0, ARTREF_LIST_ERR_ARG = 1 };

/*
 * q bf16 [batch][num_q_heads][head_dim] (QUERY_BOUND only; may be NULL
 * otherwise), k_cache bf16 pool, page_table [batch][max_pages_per_seq],
 * seq_lens [batch].  Writes block_list [batch][num_kv_heads][max_blocks_per_list],
 * block_list_len [batch][num_kv_heads] and, when `scores` is not NULL and the
 * policy is importance, scores [batch][num_kv_heads][max_blocks].
 */
int artref_block_list(const artref_list_shape* shape, const artref_list_opts* opts,
                      const uint16_t* q, const uint16_t* k_cache, const int32_t* page_table,
                      const int32_t* seq_lens, int32_t* block_list, int32_t* block_list_len,
                      double* scores, int32_t max_blocks);

#ifdef __cplusplus
}
#endif
#endif
