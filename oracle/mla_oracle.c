/*
 * mla_oracle.c -- plain CPU fp64 oracle for one decode-node mixed step.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header, table or constant with the
 * HIP library: the shapes below are restated here on purpose.
 *
 * What it computes.  The paper (section 2.3, chunked prefill; section 4.3.1,
 * Eq. 4) lets a decode node run one step over a mixed batch: B_n decode rows
 * (one new token each) plus chi - B_n rows of prefill chunks, each chunk
 * starting after a prefix that earlier chunks already cached (section 4.3.2,
 * Eq. 5: chunk i's prefix is the sum of the earlier chunk sizes).  The model it
 * serves (DeepSeek-V2-Lite, section 6) uses multi-head latent attention; in its
 * absorbed form every token caches one 576-dim latent (512 compressed dims +
 * 64 rope dims) shared by the 16 query heads, and the value is the first 512
 * latent dims.  The oracle is the plain definition of that step, in fp64, from
 * the exact bf16 inputs:
 *
 *   append:  for request r and token t in [p_r, p_r + c_r):
 *            pool[bt[r][t / P]][t % P][:] = new[cu_q[r] + t - p_r][:]
 *   attend:  row i of request r (i < c_r) sees keys j = 0 .. p_r + i of the
 *            appended pool; for each head h
 *              s_j = scale * sum_{d<576} q[row][h][d] * k_j[d]
 *              w_j = exp(s_j - max_j s_j),  l = sum_j w_j
 *              out[row][h][e] = sum_j w_j * k_j[e] / l   (e < 512)
 *              lse[row][h]    = max_j s_j + log(l)
 *
 * Keys are visited in increasing j and rows are independent, so the result
 * does not depend on the thread count.  No blocking, tiling or online
 * rescaling is used: this is the definition written out.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { OR_HEADS = 16, OR_DQK = 576, OR_DV = 512 };

static double bf16_value(uint16_t bits) {
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* Pool slot (page * P + offset) of logical key j of a request, or -1. */
static long slot_of(const int32_t *bt_row, int32_t max_pages, int32_t page_size,
                    int32_t num_pages, long j) {
    long lp = j / page_size;
    if (lp < 0 || lp >= max_pages) return -1;
    long page = bt_row[lp];
    if (page < 0 || page >= num_pages) return -1;
    return page * page_size + j % page_size;
}

int oracle_abi_version(void) { return 1; }

/* Scatter each request's new latents into its pages.  Returns 0, or -1 if a
 * slot falls outside the block table or the pool. */
int oracle_append(int32_t num_reqs, int32_t page_size, int32_t num_pages,
                  int32_t max_pages_per_req, const int32_t *q_lens,
                  const int32_t *prefix_lens, const int32_t *block_table,
                  const uint16_t *new_latents, uint16_t *pool) {
    long row0 = 0;
    for (int32_t r = 0; r < num_reqs; ++r) {
        const int32_t *bt = block_table + (long)r * max_pages_per_req;
        for (long i = 0; i < q_lens[r]; ++i) {
            long t = (long)prefix_lens[r] + i;
            long s = slot_of(bt, max_pages_per_req, page_size, num_pages, t);
            if (s < 0) return -1;
            memcpy(pool + s * OR_DQK, new_latents + (row0 + i) * OR_DQK,
                   OR_DQK * sizeof(uint16_t));
        }
        row0 += q_lens[r];
    }
    return 0;
}

/* One query row: n_keys visible keys (logical 0 .. n_keys-1) of the request
 * whose block-table row is bt_row.  out [16][512], lse [16] (may be NULL).
 * weights, if not NULL, receives [16][n_keys] softmax weights w_j / l.
 * Returns 0, or -1 on a bad slot or allocation failure. */
int oracle_attend_row(int32_t page_size, int32_t num_pages, int32_t max_pages_per_req,
                      const int32_t *bt_row, long n_keys, const uint16_t *q_row,
                      const uint16_t *pool, double scale, double *out, double *lse,
                      double *weights) {
    if (n_keys < 1) return -1;
    double *q = malloc(sizeof(double) * OR_HEADS * OR_DQK);
    double *k = malloc(sizeof(double) * OR_DQK);
    double *s = malloc(sizeof(double) * OR_HEADS * (size_t)n_keys);
    if (!q || !k || !s) { free(q); free(k); free(s); return -1; }
    for (int i = 0; i < OR_HEADS * OR_DQK; ++i) q[i] = bf16_value(q_row[i]);

    /* scores s[h][j] */
    for (long j = 0; j < n_keys; ++j) {
        long sl = slot_of(bt_row, max_pages_per_req, page_size, num_pages, j);
        if (sl < 0) { free(q); free(k); free(s); return -1; }
        for (int d = 0; d < OR_DQK; ++d) k[d] = bf16_value(pool[sl * OR_DQK + d]);
        for (int h = 0; h < OR_HEADS; ++h) {
            double acc = 0.0;
            for (int d = 0; d < OR_DQK; ++d) acc += q[h * OR_DQK + d] * k[d];
            s[h * n_keys + j] = scale * acc;
        }
    }
    /* softmax over keys, then the weighted sum of values */
    double *o = out;
    for (int h = 0; h < OR_HEADS; ++h) {
        double *sh = s + h * n_keys;
        double m = sh[0];
        for (long j = 1; j < n_keys; ++j) if (sh[j] > m) m = sh[j];
        double l = 0.0;
        for (long j = 0; j < n_keys; ++j) { sh[j] = exp(sh[j] - m); l += sh[j]; }
        for (int e = 0; e < OR_DV; ++e) o[h * OR_DV + e] = 0.0;
        for (long j = 0; j < n_keys; ++j) {
            long sl = slot_of(bt_row, max_pages_per_req, page_size, num_pages, j);
            const uint16_t *v = pool + sl * OR_DQK;
            double w = sh[j];
            for (int e = 0; e < OR_DV; ++e) o[h * OR_DV + e] += w * bf16_value(v[e]);
        }
        for (int e = 0; e < OR_DV; ++e) o[h * OR_DV + e] /= l;
        if (lse) lse[h] = m + log(l);
        if (weights)
            for (long j = 0; j < n_keys; ++j) weights[h * n_keys + j] = sh[j] / l;
    }
    free(q); free(k); free(s);
    return 0;
}

/* Request index and in-request offset of global row `row`. */
static int locate_row(int32_t num_reqs, const int32_t *q_lens, long row, int32_t *req, long *off) {
    long base = 0;
    for (int32_t r = 0; r < num_reqs; ++r) {
        if (row < base + q_lens[r]) { *req = r; *off = row - base; return 0; }
        base += q_lens[r];
    }
    return -1;
}

/* Attention for the listed global rows (rows == NULL: all rows 0..n_rows-1),
 * over a pool that already holds the step's appended latents.
 * out [n_rows][16][512], lse [n_rows][16] (may be NULL).  num_threads <= 0
 * leaves the OpenMP default.  Returns 0 or -1. */
int oracle_attend_rows(int32_t num_reqs, int32_t page_size, int32_t num_pages,
                       int32_t max_pages_per_req, const int32_t *q_lens,
                       const int32_t *prefix_lens, const int32_t *block_table,
                       const uint16_t *q, const uint16_t *pool, double scale,
                       long n_rows, const int64_t *rows, double *out, double *lse,
                       int32_t num_threads) {
    int status = 0;
#ifdef _OPENMP
    if (num_threads > 0) omp_set_num_threads(num_threads);
#else
    (void)num_threads;
#endif
#pragma omp parallel for schedule(dynamic, 1) reduction(| : status)
    for (long n = 0; n < n_rows; ++n) {
        long row = rows ? rows[n] : n;
        int32_t r;
        long i;
        if (locate_row(num_reqs, q_lens, row, &r, &i) != 0) { status |= 1; continue; }
        long n_keys = (long)prefix_lens[r] + i + 1;
        int rc = oracle_attend_row(page_size, num_pages, max_pages_per_req,
                                   block_table + (long)r * max_pages_per_req, n_keys,
                                   q + row * OR_HEADS * OR_DQK, pool, scale,
                                   out + n * OR_HEADS * OR_DV, lse ? lse + n * OR_HEADS : NULL,
                                   NULL);
        if (rc != 0) status |= 1;
    }
    return status ? -1 : 0;
}

int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
