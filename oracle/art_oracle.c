/*
 * art_oracle.c -- fp64 CPU oracle for ART decode attention.
 *
 * TEST INFRASTRUCTURE ONLY (see art_oracle.h).  Plain, slow and written to be
 * checked against the paper by eye; it is never called by the product path.
 *
 * Paper passages followed:
 *   Eq. (1), Sec. 3.1 ......... O = softmax(Q K^T / sqrt(d)) V; the scale is
 *                               passed in (the fp32 value the kernel gets).
 *   Sec. 3.1 + Appendix A ..... blocks processed in sequence; per block t the
 *                               block output u(t) = softmax(q K_t^T s) V_t and
 *                               mass l(t) = sum_k exp(s q.k), A(t) = sum l(j),
 *                               o(t) = (A(t-1) o(t-1) + l(t) u(t)) / A(t).
 *                               Computed in the log domain (ln l, ln A) so that
 *                               no exponential overflows; the coefficients
 *                               A(t-1)/A(t) and l(t)/A(t) are the same numbers.
 *   Eq. (2), Sec. 3.2 ......... d_scale = ||x(t) - x(t-1)||_2,
 *                               d_direction = 1 - cos(x(t), x(t-1)),
 *                               x(t) = P o(t) (the probe of Appendix A).
 *   Sec. 3.2 .................. stable iff d_scale < tau and d_direction < phi.
 *   Eq. (3) ................... c(t) = c(t-1) + 1 if stable else 0.
 *   Algorithm 1 ............... o(0) = 0, c(0) = 0; after the update of step t,
 *                               break once c(t) >= p; return o(t).
 *   Sec. 3.4 .................. full-KV traversal is recency-first (reverse
 *                               temporal order); importance-first traversal
 *                               follows a supplied list of block ids.
 *
 * Readings where the paper is silent or ambiguous:
 *   R1 probe: by default x(t) is the whole normalised output o(t) of each
 *      query head (P = I, the full-output detector Appendix B compares
 *      against).  With probe_stride s > 1, P keeps the coordinates
 *      0, s, 2s, ... of o(t) (m = D / s): a fixed subsample spread over the
 *      head dimension, in place of Sec. 3.2's subsample taken from the
 *      accumulator's register layout (m = 32 there, i.e. s = 4 at D = 128).
 *   R2 o(t) is the normalised running output (Appendix A), not the
 *      unnormalised accumulator.  With scale_of_accumulator set, d_scale is
 *      taken instead on X(t) = l(t) o(t), the accumulator Algorithm 1 carries
 *      before its final normalisation: l(t) = sum over the consumed tokens of
 *      exp(s - m(t)), m(t) the running maximum score, each X in its own
 *      step's reference (no rescaling of X(t-1)).  d_direction is the same
 *      either way (l > 0 does not change a cosine).
 *   R3 grouped-query attention: one decision per (sequence, KV head); a step is
 *      stable only if it is stable for every query head of the group.  With
 *      per_head_stop set, each query head instead runs its own counter and
 *      stops on its own (its output and lse are those of its stop); the group
 *      reads blocks until its last head has stopped.
 *   R4 step 1 compares against o(0) = 0: cos is 0/0, the comparison is false,
 *      so step 1 is never stable.  Generally, a zero-norm vector makes the step
 *      unstable.
 *   R5 strict "<" as in Algorithm 1 (Definition 2 of Appendix A uses <=).
 *   R6 the block that triggers the break is included: stop_block = t* is the
 *      number of blocks consumed; out = o(t*).  Without a break t* = T.
 *   R7 lse = ln A(t*), over the tokens of the consumed blocks only.
 *   R8 a partial last block holds tokens [blk*Bk, L); block ids in a list must
 *      lie in [0, ceil(L/Bk)) and be unique; T = 0 gives out = 0,
 *      lse = -inf, stop_block = 0.
 */
#include "art_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double bf16_to_double(uint16_t bits) {
    uint32_t w = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

static double log_add_exp(double a, double b) {
    if (a == -INFINITY) return b;
    if (b == -INFINITY) return a;
    double m = a > b ? a : b;
    return m + log(exp(a - m) + exp(b - m));
}

/* group (b, kvh); returns 0 or an ARTREF_ERR_* code */
static int run_group(const artref_shape* S, const artref_opts* O, int b, int kvh,
                     const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                     const int32_t* page_table, const int32_t* seq_lens,
                     const int32_t* block_list, const int32_t* block_list_len,
                     const int32_t* force_stop, double* out, double* lse,
                     int32_t* stop_block, int32_t* head_stop, double* trace,
                     int32_t trace_steps) {
    const int g = S->num_q_heads / S->num_kv_heads;
    const int D = S->head_dim;
    const int Bk = S->block_size;
    const int ps = O->probe_stride;
    const int L = seq_lens[b];
    const int nblk = L > 0 ? (L + Bk - 1) / Bk : 0;
    const int gi = b * S->num_kv_heads + kvh;
    int rc = ARTREF_OK;

    /* traversal list (Sec. 3.4) */
    int T;
    int* list = NULL;
    if (block_list) {
        const int row = S->list_per_head ? gi : b;
        T = block_list_len[row];
        if (T < 0 || T > S->max_blocks_per_list) return ARTREF_ERR_ARG;
        list = (int*)malloc(sizeof(int) * (T > 0 ? T : 1));
        char* seen = (char*)calloc(nblk > 0 ? nblk : 1, 1);
        for (int i = 0; i < T; ++i) {
            int id = block_list[(int64_t)row * S->max_blocks_per_list + i];
            if (id < 0 || id >= nblk || seen[id]) { rc = ARTREF_ERR_INDEX; break; }
            seen[id] = 1;
            list[i] = id;
        }
        free(seen);
        if (rc) { free(list); return rc; }
    } else {
        T = nblk;
        list = (int*)malloc(sizeof(int) * (T > 0 ? T : 1));
        for (int i = 0; i < T; ++i)
            list[i] = (O->dense_order == 1) ? i : (nblk - 1 - i);
    }

    double* qd   = (double*)malloc(sizeof(double) * g * D);
    double* o    = (double*)calloc((size_t)g * D, sizeof(double));  /* o(0) = 0 */
    double* onew = (double*)malloc(sizeof(double) * g * D);
    double* u    = (double*)malloc(sizeof(double) * g * D);
    double* s    = (double*)malloc(sizeof(double) * g * Bk);
    double* logA = (double*)malloc(sizeof(double) * g);
    double* mrun = (double*)malloc(sizeof(double) * g);             /* running max score */
    for (int i = 0; i < g; ++i) {
        logA[i] = -INFINITY;                                         /* A(0) = 0 */
        mrun[i] = -INFINITY;
        const uint16_t* qh = q + ((int64_t)b * S->num_q_heads + kvh * g + i) * D;
        for (int d = 0; d < D; ++d) qd[i * D + d] = bf16_to_double(qh[d]);
    }
    const int per_head = O->per_head_stop;
    int fstop = (force_stop && !per_head) ? force_stop[gi] : 0;
    int c = 0;      /* patience counter, Eq. (3) */
    int tstar = T;  /* no break: all T blocks consumed */
    /* R3 variant: a counter and a stop per query head (0 = still reading) */
    int* ch = (int*)calloc(g, sizeof(int));
    int* hstop = (int*)calloc(g, sizeof(int));
    int running = g;

    for (int t = 1; t <= T && !rc; ++t) {
        const int blk = list[t - 1];
        const int j0 = blk * Bk;
        const int j1 = (j0 + Bk < L) ? j0 + Bk : L;
        const int n = j1 - j0;
        /* scores s_hj = scale * q_h . k_j, fp64 from the exact bf16 values */
        for (int j = 0; j < n; ++j) {
            const int tok = j0 + j;
            const int32_t page = page_table[(int64_t)b * S->max_pages_per_seq + tok / S->page_size];
            if (page < 0 || page >= S->num_pages) { rc = ARTREF_ERR_INDEX; break; }
            const uint16_t* kj = kc + page * S->k_stride_page + kvh * S->k_stride_head
                                 + (int64_t)(tok % S->page_size) * S->k_stride_token;
            for (int i = 0; i < g; ++i) {
                double dot = 0.0;
                for (int d = 0; d < D; ++d) dot += qd[i * D + d] * bf16_to_double(kj[d]);
                s[i * Bk + j] = O->scale * dot;
            }
        }
        if (rc) break;
        int all_stable = 1;
        for (int i = 0; i < g; ++i) {
            /* block softmax output u(t) and block mass ln l(t) (Appendix A) */
            double mb = -INFINITY;
            for (int j = 0; j < n; ++j) if (s[i * Bk + j] > mb) mb = s[i * Bk + j];
            double ssum = 0.0;
            for (int d = 0; d < D; ++d) u[i * D + d] = 0.0;
            for (int j = 0; j < n; ++j) {
                const int tok = j0 + j;
                const int32_t page = page_table[(int64_t)b * S->max_pages_per_seq + tok / S->page_size];
                const uint16_t* vj = vc + page * S->v_stride_page + kvh * S->v_stride_head
                                     + (int64_t)(tok % S->page_size) * S->v_stride_token;
                const double e = exp(s[i * Bk + j] - mb);
                ssum += e;
                for (int d = 0; d < D; ++d) u[i * D + d] += e * bf16_to_double(vj[d]);
            }
            for (int d = 0; d < D; ++d) u[i * D + d] /= ssum;
            const double logl = mb + log(ssum);
            const double logA_new = log_add_exp(logA[i], logl);
            const double keep = exp(logA[i] - logA_new);   /* A(t-1) / A(t) */
            /* R2 variant: accumulator weights l(t-1), l(t) in their own references */
            const double m_new = mb > mrun[i] ? mb : mrun[i];
            const double l_old = (logA[i] == -INFINITY) ? 0.0 : exp(logA[i] - mrun[i]);
            const double l_new = exp(logA_new - m_new);
            const double xs_new = O->scale_of_accumulator ? l_new : 1.0;
            const double xs_old = O->scale_of_accumulator ? l_old : 1.0;
            mrun[i] = m_new;
            const double w = exp(logl - logA_new);         /* l(t) / A(t)   */
            logA[i] = logA_new;
            /* o(t) = (A(t-1) o(t-1) + l(t) u(t)) / A(t) */
            for (int d = 0; d < D; ++d)
                onew[i * D + d] = keep * o[i * D + d] + w * u[i * D + d];
            /* probe coordinates of o(t) and o(t-1) (R1) */
            double ds2 = 0.0, dot = 0.0, n_new = 0.0, n_old = 0.0;
            for (int d = 0; d < D; d += ps) {
                const double x = onew[i * D + d], x0 = o[i * D + d];
                const double diff = xs_new * x - xs_old * x0;
                ds2 += diff * diff;
                dot += x * x0;
                n_new += x * x;
                n_old += x0 * x0;
            }
            /* Eq. (2) */
            const double d_scale = sqrt(ds2);
            const double d_dir = (n_new > 0.0 && n_old > 0.0)
                                     ? 1.0 - dot / (sqrt(n_new) * sqrt(n_old))
                                     : NAN;   /* R4: undefined cosine */
            /* Sec. 3.2 (R3: every head of the group must be stable) */
            const int stable = (d_scale < O->tau) && (d_dir < O->phi);
            if (!stable) all_stable = 0;
            if (per_head && !hstop[i]) {
                /* Eq. (3) and the break of Algorithm 1 for this head alone */
                ch[i] = stable ? ch[i] + 1 : 0;
                const int fh = force_stop ? force_stop[(int64_t)b * S->num_q_heads + kvh * g + i] : 0;
                if ((fh >= 1) ? (t >= fh) : (ch[i] >= O->patience)) {
                    hstop[i] = t;
                    --running;
                    const int h = kvh * g + i;
                    double* oh = out + ((int64_t)b * S->num_q_heads + h) * D;
                    for (int d = 0; d < D; ++d) oh[d] = keep * o[i * D + d] + w * u[i * D + d];
                    lse[(int64_t)b * S->num_q_heads + h] = logA[i];
                }
            }
            if (trace && t <= trace_steps) {
                double* tr = trace + (((int64_t)gi * trace_steps + (t - 1)) * g + i) * 2;
                tr[0] = d_scale;
                tr[1] = d_dir;
            }
        }
        memcpy(o, onew, sizeof(double) * g * D);
        if (per_head) {
            if (running == 0) { tstar = t; break; }
            continue;
        }
        c = all_stable ? c + 1 : 0;                    /* Eq. (3) */
        if (fstop >= 1) {
            if (t >= fstop) { tstar = t; break; }
        } else if (c >= O->patience) {               /* Algorithm 1: break */
            tstar = t;
            break;
        }
    }
    if (!rc) {
        for (int i = 0; i < g; ++i) {
            const int h = kvh * g + i;
            if (per_head && hstop[i]) {       /* written at the head's own stop */
                if (head_stop) head_stop[(int64_t)b * S->num_q_heads + h] = hstop[i];
                continue;
            }
            double* oh = out + ((int64_t)b * S->num_q_heads + h) * D;
            for (int d = 0; d < D; ++d) oh[d] = (T > 0) ? o[i * D + d] : 0.0;
            lse[(int64_t)b * S->num_q_heads + h] = (T > 0) ? logA[i] : -INFINITY;
            if (head_stop) head_stop[(int64_t)b * S->num_q_heads + h] = (T > 0) ? tstar : 0;
        }
        stop_block[gi] = (T > 0) ? tstar : 0;
        if (trace) {
            for (int t = (T < trace_steps ? T : trace_steps) + 1; t <= trace_steps; ++t)
                for (int i = 0; i < g; ++i) {
                    double* tr = trace + (((int64_t)gi * trace_steps + (t - 1)) * g + i) * 2;
                    tr[0] = NAN;
                    tr[1] = NAN;
                }
            /* steps after the break were not evaluated */
            for (int t = tstar + 1; t <= (T < trace_steps ? T : trace_steps); ++t)
                for (int i = 0; i < g; ++i) {
                    double* tr = trace + (((int64_t)gi * trace_steps + (t - 1)) * g + i) * 2;
                    tr[0] = NAN;
                    tr[1] = NAN;
                }
        }
    }
    free(list); free(qd); free(o); free(onew); free(u); free(s); free(logA); free(mrun);
    free(ch); free(hstop);
    return rc;
}

int artref_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

int artref_decode(const artref_shape* S, const artref_opts* O,
                  const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                  const int32_t* page_table, const int32_t* seq_lens,
                  const int32_t* block_list, const int32_t* block_list_len,
                  const int32_t* force_stop, const uint8_t* group_mask,
                  double* out, double* lse, int32_t* stop_block, int32_t* head_stop,
                  double* trace, int32_t trace_steps,
                  int32_t num_threads, int32_t* err_group) {
    if (err_group) *err_group = -1;
    if (!S || !O || !q || !k_cache || !v_cache || !page_table || !seq_lens || !out ||
        !lse || !stop_block)
        return ARTREF_ERR_ARG;
    if (S->batch < 0 || S->num_kv_heads <= 0 || S->num_q_heads <= 0 ||
        S->num_q_heads % S->num_kv_heads || S->head_dim <= 0 || S->block_size <= 0 ||
        S->page_size <= 0 || O->patience < 1 || O->probe_stride < 1 ||
        S->head_dim % O->probe_stride || (block_list && !block_list_len) ||
        (!block_list && block_list_len) || (trace && trace_steps < 0))
        return ARTREF_ERR_ARG;
    for (int b = 0; b < S->batch; ++b)
        if (seq_lens[b] < 0 || seq_lens[b] > (int64_t)S->max_pages_per_seq * S->page_size)
            return ARTREF_ERR_ARG;
    const int ngroups = S->batch * S->num_kv_heads;
    int first_err = ngroups, err_code = ARTREF_OK;
#ifdef _OPENMP
    if (num_threads > 0) omp_set_num_threads(num_threads);
#pragma omp parallel for schedule(dynamic, 1)
#endif
    for (int gi = 0; gi < ngroups; ++gi) {
        if (group_mask && !group_mask[gi]) continue;
        const int b = gi / S->num_kv_heads, kvh = gi % S->num_kv_heads;
        int rc = run_group(S, O, b, kvh, q, k_cache, v_cache, page_table, seq_lens,
                           block_list, block_list_len, force_stop, out, lse, stop_block,
                           head_stop, trace, trace_steps);
        if (rc) {
#ifdef _OPENMP
#pragma omp critical
#endif
            {
                if (gi < first_err) { first_err = gi; err_code = rc; }
            }
        }
    }
    if (err_code != ARTREF_OK && err_group) *err_group = first_err;
    return err_code;
}
