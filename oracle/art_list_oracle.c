/*
 * art_list_oracle.c -- fp64 CPU oracle for ART's traversal lists.
 *
 * TEST INFRASTRUCTURE ONLY (like art_oracle.c): the plain statement of the
 * lists the GPU list producer must build.  Never called by the product path;
 * shares no code with the HIP library.
 *
 * Sec. 3.4 composes the termination with the traversal order of the base KV
 * policy:
 *   - full KV cache: reverse temporal order (built into the decode call);
 *   - pattern-based policies (a StreamingLLM-style cache of sink tokens plus
 *     a recent window): recency-first over the retained blocks while the
 *     sink blocks are kept;
 *   - policies with importance scores per block: the selected blocks in
 *     descending order of score, handed to the kernel as an index list.
 *
 * Readings (the paper names the orders, not the scores or the selection):
 *   L1 block scores (two kinds, both computed in fp64 with the sum taken in
 *      increasing dimension order, so that any implementation that keeps
 *      that order gets the same bits):
 *        KEY_NORM:    s_i = max over the block's tokens j of sum_d k_jd^2
 *                     (the squared largest key norm; same order as the norm);
 *        QUERY_BOUND: s_i = max over the group's query heads h of
 *                     sum_d max(q_hd * min_j k_jd, q_hd * max_j k_jd),
 *                     an upper bound of q_h . k_j over the block's tokens.
 *      Tokens at or beyond the sequence length are not part of a block.
 *   L2 importance selection: the first `sink_blocks` blocks and (keep_last)
 *      the last block are always selected; of the other blocks, the
 *      budget - (forced count) with the largest scores are added (equal
 *      scores: smaller block id first).  The list holds the selected blocks
 *      in descending score order (equal scores: smaller id first).
 *   L3 streaming list: blocks 0 .. sink_blocks-1 in increasing order (the
 *      kept sinks are visited first, so that a stop never drops them), then
 *      the `budget` most recent other blocks, newest first.
 *   L4 an empty sequence gives an empty list.
 */
#include "art_list_oracle.h"

#include <stdlib.h>
#include <string.h>

static double bf16(uint16_t bits) {
    uint32_t w = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

static const uint16_t* key_row(const artref_list_shape* S, const uint16_t* kc, const int32_t* page_table,
                               int b, int kvh, int tok) {
    const int32_t page = page_table[(int64_t)b * S->max_pages_per_seq + tok / S->page_size];
    return kc + page * S->k_stride_page + kvh * S->k_stride_head +
           (int64_t)(tok % S->page_size) * S->k_stride_token;
}

/* L1 */
static double block_score(const artref_list_shape* S, int kind, const uint16_t* q, const uint16_t* kc,
                          const int32_t* page_table, int b, int kvh, int blk, int L) {
    const int D = S->head_dim, Bk = S->block_size;
    const int g = S->num_q_heads / S->num_kv_heads;
    const int j0 = blk * Bk, j1 = (j0 + Bk < L) ? j0 + Bk : L;
    if (kind == ARTREF_SCORE_KEY_NORM) {
        double best = 0.0;
        for (int j = j0; j < j1; ++j) {
            const uint16_t* k = key_row(S, kc, page_table, b, kvh, j);
            double s = 0.0;
            for (int d = 0; d < D; ++d) s += bf16(k[d]) * bf16(k[d]);
            if (j == j0 || s > best) best = s;
        }
        return best;
    }
    /* QUERY_BOUND: channel-wise extremes of the block's keys */
    double* kmin = malloc(sizeof(double) * D);
    double* kmax = malloc(sizeof(double) * D);
    if (!kmin || !kmax) { free(kmin); free(kmax); return 0.0; }
    for (int j = j0; j < j1; ++j) {
        const uint16_t* k = key_row(S, kc, page_table, b, kvh, j);
        for (int d = 0; d < D; ++d) {
            const double x = bf16(k[d]);
            if (j == j0 || x < kmin[d]) kmin[d] = x;
            if (j == j0 || x > kmax[d]) kmax[d] = x;
        }
    }
    double best = 0.0;
    for (int i = 0; i < g; ++i) {
        const uint16_t* qh = q + ((int64_t)b * S->num_q_heads + kvh * g + i) * D;
        double s = 0.0;
        for (int d = 0; d < D; ++d) {
            const double a = bf16(qh[d]) * kmin[d], c = bf16(qh[d]) * kmax[d];
            s += a > c ? a : c;
        }
        if (i == 0 || s > best) best = s;
    }
    free(kmin);
    free(kmax);
    return best;
}

typedef struct { double s; int id; } scored;

/* descending score, then ascending id */
static int by_score(const void* a, const void* b) {
    const scored* x = a;
    const scored* y = b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->id > y->id) - (x->id < y->id);
}

int artref_block_list(const artref_list_shape* S, const artref_list_opts* O, const uint16_t* q,
                      const uint16_t* k_cache, const int32_t* page_table, const int32_t* seq_lens,
                      int32_t* block_list, int32_t* block_list_len, double* scores, int32_t max_blocks) {
    if (!S || !O || !k_cache || !page_table || !seq_lens || !block_list || !block_list_len)
        return ARTREF_LIST_ERR_ARG;
    if (S->num_kv_heads <= 0 || S->num_q_heads % S->num_kv_heads || S->block_size <= 0 ||
        S->page_size <= 0 || O->budget < 0 || O->sink_blocks < 0 ||
        (O->policy != ARTREF_LIST_IMPORTANCE && O->policy != ARTREF_LIST_STREAMING) ||
        (O->policy == ARTREF_LIST_IMPORTANCE && O->score_kind != ARTREF_SCORE_KEY_NORM &&
         O->score_kind != ARTREF_SCORE_QUERY_BOUND) ||
        (O->policy == ARTREF_LIST_IMPORTANCE && O->score_kind == ARTREF_SCORE_QUERY_BOUND && !q))
        return ARTREF_LIST_ERR_ARG;
    for (int b = 0; b < S->batch; ++b) {
        const int L = seq_lens[b];
        if (L < 0 || L > (int64_t)S->max_pages_per_seq * S->page_size) return ARTREF_LIST_ERR_ARG;
        const int n = L > 0 ? (L + S->block_size - 1) / S->block_size : 0;
        if (n > max_blocks) return ARTREF_LIST_ERR_ARG;
        for (int kvh = 0; kvh < S->num_kv_heads; ++kvh) {
            const int gi = b * S->num_kv_heads + kvh;
            int32_t* out = block_list + (int64_t)gi * S->max_blocks_per_list;
            int len = 0;
            if (O->policy == ARTREF_LIST_STREAMING) {
                /* L3 */
                const int ns = O->sink_blocks < n ? O->sink_blocks : n;
                for (int i = 0; i < ns; ++i) {
                    if (len >= S->max_blocks_per_list) return ARTREF_LIST_ERR_ARG;
                    out[len++] = i;
                }
                for (int i = n - 1, taken = 0; i >= ns && taken < O->budget; --i, ++taken) {
                    if (len >= S->max_blocks_per_list) return ARTREF_LIST_ERR_ARG;
                    out[len++] = i;
                }
                block_list_len[gi] = len;
                continue;
            }
            /* L1: score every block of the sequence */
            scored* all = malloc(sizeof(scored) * (n > 0 ? n : 1));
            if (!all) return ARTREF_LIST_ERR_ARG;
            for (int i = 0; i < n; ++i) {
                all[i].id = i;
                all[i].s = block_score(S, O->score_kind, q, k_cache, page_table, b, kvh, i, L);
                if (scores) scores[(int64_t)gi * max_blocks + i] = all[i].s;
            }
            /* L2: forced blocks, then the best others */
            char* forced = calloc(n > 0 ? n : 1, 1);
            if (!forced) { free(all); return ARTREF_LIST_ERR_ARG; }
            int nf = 0;
            for (int i = 0; i < n && i < O->sink_blocks; ++i) { forced[i] = 1; ++nf; }
            if (O->keep_last && n > 0 && !forced[n - 1]) { forced[n - 1] = 1; ++nf; }
            qsort(all, n, sizeof(scored), by_score);
            int others = O->budget - nf;
            for (int r = 0; r < n; ++r) {
                const int id = all[r].id;
                int take = forced[id];
                if (!take && others > 0) { take = 1; --others; }
                if (take) {
                    if (len >= S->max_blocks_per_list) { free(all); free(forced); return ARTREF_LIST_ERR_ARG; }
                    out[len++] = id;
                }
            }
            block_list_len[gi] = len;
            free(all);
            free(forced);
        }
    }
    return ARTREF_LIST_OK;
}
