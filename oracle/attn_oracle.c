/*
 * Plain fp64 CPU oracle for one attention call over a mixed batch of block
 * decodes and whole prefills (cached diffusion-LLM serving).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing on the product path links, loads or calls
 * this file; only the tests, the smoke check and the benchmark's CPU-baseline
 * leg do. It shares no code, header, table or helper with the HIP library.
 *
 * What it computes (the plain definition; the method reaches it exactly up to
 * rounding):
 *   - dLLM attention is full bidirectional attention over prompt + response:
 *     the causal mask is dropped (Sec. 2.1), so every query row of an item
 *     attends to every position [0, L) of that item.
 *   - A block decode reuses the approximately cached KV of its request and
 *     recomputes only its own block (Sec. 2.2, blockwise Fast-dLLM cache):
 *     positions [o, o+n) take the fresh rows k_new / v_new, all others come
 *     from the cache as it stood before the call.
 *   - A per-token cached decode (Sec. 2.2, the dKV-Cache-PD variant: prompt
 *     KV fixed, response tokens refreshed individually) recomputes an
 *     arbitrary set of positions: when a position list q_pos is given, row r
 *     of an item sits at position q_pos[r] instead of o + r; every other rule
 *     is the same.
 *   - A prefill brings its whole sequence as fresh rows (o = 0, n = L) and
 *     refreshes the cache with them (Sec. 2.2; whole, never chunked, Sec. 3.2).
 *   - Per (item, query row r, query head h), with G = Hq / Hkv and the KV head
 *     g = floor(h / G) (contiguous query-head groups):
 *         s_j = sigma * sum_d q[r,h,d] * Khat[j,g,d]         j in [0, L)
 *         m = max_j s_j,  w_j = exp(s_j - m),  Z = sum_j w_j
 *         o[r,h,:] = sum_j w_j Vhat[j,g,:] / Z,  lse[r,h] = m + ln Z
 *     sigma is the float32 softmax scale widened to double.
 * Inputs are bf16 bit patterns; each is widened exactly to double.
 *
 * Parity pins for every function here live in tests/test_oracle.py (brute
 * force in exact rationals, torch float64 SDPA, closed forms, invariants).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_EINVAL -1
#define ORACLE_ENOMEM -2

/* bf16 -> double: bf16 is the top 16 bits of an IEEE binary32 */
static double widen(uint16_t h)
{
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

typedef struct {
    int32_t n_items, hq, hkv, d;
    const int32_t *q_indptr, *q_offset, *q_pos, *kv_len;
    const int64_t *ctx_indptr;
    const uint16_t *q, *k_new, *v_new, *k_ctx, *v_ctx;
    /* fresh[seq_base[i] + j]: packed row that holds position j of item i, or
     * -1 when position j comes from the pre-call cache */
    int64_t *seq_base, *fresh;
} call_t;

/* position of local row r of item i */
static int64_t row_pos(const call_t *c, int32_t i, int64_t r)
{
    return c->q_pos ? c->q_pos[c->q_indptr[i] + r] : c->q_offset[i] + r;
}

/*
 * Row j (position in [0, L)) of the assembled key (or value) sequence of item
 * i for KV head g: the fresh row that sits at position j, else the pre-call
 * cache.
 */
static const uint16_t *seq_row(const call_t *c, int32_t i, int64_t j, int32_t g, int value)
{
    int64_t row = c->fresh[c->seq_base[i] + j];
    if (row >= 0) {
        const uint16_t *base = value ? c->v_new : c->k_new;
        return base + (row * c->hkv + g) * c->d;
    }
    const uint16_t *base = value ? c->v_ctx : c->k_ctx;
    row = c->ctx_indptr[i] + j;
    return base + (row * c->hkv + g) * c->d;
}

static void release(call_t *c)
{
    free(c->seq_base);
    free(c->fresh);
    c->seq_base = c->fresh = NULL;
}

/* validate the call and build the position -> fresh row map */
static int check_call(call_t *c)
{
    c->seq_base = c->fresh = NULL;
    if (c->n_items < 0 || c->hq <= 0 || c->hkv <= 0 || c->d <= 0)
        return ORACLE_EINVAL;
    if (c->hq % c->hkv != 0)
        return ORACLE_EINVAL;
    int64_t total = 0;
    for (int32_t i = 0; i < c->n_items; ++i) {
        int64_t n = (int64_t)c->q_indptr[i + 1] - c->q_indptr[i];
        int64_t L = c->kv_len[i];
        int64_t ctx = c->ctx_indptr[i + 1] - c->ctx_indptr[i];
        if (n < 1 || L < 1)
            return ORACLE_EINVAL;
        /* positions strictly increasing inside [0, L) */
        for (int64_t r = 0; r < n; ++r) {
            int64_t p = row_pos(c, i, r);
            if (p < 0 || p >= L || (r > 0 && p <= row_pos(c, i, r - 1)))
                return ORACLE_EINVAL;
        }
        /* an item without pre-call context must bring every row fresh */
        if (ctx == 0 && n != L)
            return ORACLE_EINVAL;
        if (ctx != 0 && ctx != L)
            return ORACLE_EINVAL;
        total += L;
    }
    c->seq_base = (int64_t *)malloc(sizeof(int64_t) * (size_t)(c->n_items + 1));
    c->fresh = (int64_t *)malloc(sizeof(int64_t) * (size_t)(total > 0 ? total : 1));
    if (!c->seq_base || !c->fresh) {
        release(c);
        return ORACLE_ENOMEM;
    }
    c->seq_base[0] = 0;
    for (int32_t i = 0; i < c->n_items; ++i) {
        int64_t base = c->seq_base[i], L = c->kv_len[i];
        for (int64_t j = 0; j < L; ++j)
            c->fresh[base + j] = -1;
        for (int64_t r = 0; r < (int64_t)c->q_indptr[i + 1] - c->q_indptr[i]; ++r)
            c->fresh[base + row_pos(c, i, r)] = (int64_t)c->q_indptr[i] + r;
        c->seq_base[i + 1] = base + L;
    }
    return ORACLE_OK;
}

/* Scores, weights and output of one (item, row, head); w has room for L. */
static void one_row(const call_t *c, double sigma, int32_t i, int64_t r_global, int32_t h,
                    double *w, double *out, double *lse)
{
    const int32_t G = c->hq / c->hkv;
    const int32_t g = h / G;
    const int64_t L = c->kv_len[i];
    const uint16_t *qrow = c->q + (r_global * c->hq + h) * c->d;

    double m = -INFINITY;
    for (int64_t j = 0; j < L; ++j) {
        const uint16_t *krow = seq_row(c, i, j, g, 0);
        double dot = 0.0;
        for (int32_t e = 0; e < c->d; ++e)
            dot += widen(qrow[e]) * widen(krow[e]);
        w[j] = sigma * dot;
        if (w[j] > m)
            m = w[j];
    }
    double Z = 0.0;
    for (int64_t j = 0; j < L; ++j) {
        w[j] = exp(w[j] - m);
        Z += w[j];
    }
    if (out) {
        for (int32_t e = 0; e < c->d; ++e)
            out[e] = 0.0;
        for (int64_t j = 0; j < L; ++j) {
            const uint16_t *vrow = seq_row(c, i, j, g, 1);
            for (int32_t e = 0; e < c->d; ++e)
                out[e] += w[j] * widen(vrow[e]);
        }
        for (int32_t e = 0; e < c->d; ++e)
            out[e] /= Z;
    }
    if (lse)
        *lse = m + log(Z);
    /* leave normalized weights in w for the debug entry */
    for (int64_t j = 0; j < L; ++j)
        w[j] /= Z;
}

/* item index of a packed query row (binary search over q_indptr) */
static int32_t item_of_row(const call_t *c, int64_t r)
{
    int32_t lo = 0, hi = c->n_items - 1;
    while (lo < hi) {
        int32_t mid = (lo + hi + 1) / 2;
        if (c->q_indptr[mid] <= r)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

/*
 * Attention outputs for a selection of (packed row, head) pairs.
 *
 * q [sum n, hq, d], k_new / v_new [sum n, hkv, d]: bf16 bits, packed by item.
 * k_ctx / v_ctx: bf16 bits, the logical (unpaged) pre-call cache content of
 *   every item, rows [ctx_indptr[i], ctx_indptr[i+1]) for item i, each row
 *   [hkv, d]. An item with no context (a prefill) has an empty range.
 * sel: n_sel entries (packed_row * hq + head); NULL means every pair in order.
 * out: [n_sel, d] doubles; lse: [n_sel] doubles (either may be NULL).
 * Returns 0, or a negative code for an invalid call.
 */
int oracle_attn(int32_t n_items, int32_t hq, int32_t hkv, int32_t d, float sm_scale,
                const int32_t *q_indptr, const int32_t *q_offset, const int32_t *q_pos,
                const int32_t *kv_len, const int64_t *ctx_indptr, const uint16_t *q,
                const uint16_t *k_new, const uint16_t *v_new, const uint16_t *k_ctx,
                const uint16_t *v_ctx, const int64_t *sel, int64_t n_sel, double *out, double *lse)
{
    call_t c = {n_items, hq, hkv, d, q_indptr, q_offset, q_pos, kv_len, ctx_indptr,
                q, k_new, v_new, k_ctx, v_ctx, NULL, NULL};
    int rc = check_call(&c);
    if (rc)
        return rc;
    const int64_t total_rows = n_items ? q_indptr[n_items] : 0;
    const int64_t count = sel ? n_sel : total_rows * hq;
    int64_t max_l = 1;
    for (int32_t i = 0; i < n_items; ++i)
        if (kv_len[i] > max_l)
            max_l = kv_len[i];
    for (int64_t s = 0; sel && s < count; ++s)
        if (sel[s] < 0 || sel[s] >= total_rows * hq) {
            release(&c);
            return ORACLE_EINVAL;
        }
    const double sigma = (double)sm_scale;
    int failed = 0;

#pragma omp parallel
    {
        double *w = (double *)malloc(sizeof(double) * (size_t)max_l);
        if (!w) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 4)
        for (int64_t s = 0; s < count; ++s) {
            if (!w)
                continue;
            int64_t pair = sel ? sel[s] : s;
            int64_t r = pair / hq;
            int32_t h = (int32_t)(pair % hq);
            int32_t i = item_of_row(&c, r);
            one_row(&c, sigma, i, r, h, w, out ? out + s * d : NULL, lse ? lse + s : NULL);
        }
        free(w);
    }
    release(&c);
    return failed ? ORACLE_ENOMEM : ORACLE_OK;
}

/*
 * Normalized softmax weights w_j / Z, j in [0, L), of one (packed row, head).
 * w_out must hold kv_len of the row's item.
 */
int oracle_weights(int32_t n_items, int32_t hq, int32_t hkv, int32_t d, float sm_scale,
                   const int32_t *q_indptr, const int32_t *q_offset, const int32_t *q_pos,
                   const int32_t *kv_len, const int64_t *ctx_indptr, const uint16_t *q,
                   const uint16_t *k_new, const uint16_t *v_new, const uint16_t *k_ctx,
                   const uint16_t *v_ctx, int64_t row, int32_t head, double *w_out)
{
    call_t c = {n_items, hq, hkv, d, q_indptr, q_offset, q_pos, kv_len, ctx_indptr,
                q, k_new, v_new, k_ctx, v_ctx, NULL, NULL};
    int rc = check_call(&c);
    if (rc)
        return rc;
    if (row < 0 || row >= q_indptr[n_items] || head < 0 || head >= hq) {
        release(&c);
        return ORACLE_EINVAL;
    }
    int32_t i = item_of_row(&c, row);
    one_row(&c, (double)sm_scale, i, row, head, w_out, NULL, NULL);
    release(&c);
    return ORACLE_OK;
}

/*
 * The cache content of item i after the call: positions [0, L) with the fresh
 * rows written over their positions. k_out / v_out: [L, hkv, d] bf16 bits.
 */
int oracle_expected_kv(int32_t n_items, int32_t hkv, int32_t d, const int32_t *q_indptr,
                       const int32_t *q_offset, const int32_t *q_pos, const int32_t *kv_len,
                       const int64_t *ctx_indptr, const uint16_t *k_new, const uint16_t *v_new,
                       const uint16_t *k_ctx, const uint16_t *v_ctx, int32_t item, uint16_t *k_out,
                       uint16_t *v_out)
{
    call_t c = {n_items, hkv, hkv, d, q_indptr, q_offset, q_pos, kv_len, ctx_indptr,
                NULL, k_new, v_new, k_ctx, v_ctx, NULL, NULL};
    int rc = check_call(&c);
    if (rc)
        return rc;
    if (item < 0 || item >= n_items) {
        release(&c);
        return ORACLE_EINVAL;
    }
    for (int64_t j = 0; j < kv_len[item]; ++j)
        for (int32_t g = 0; g < hkv; ++g) {
            memcpy(k_out + (j * hkv + g) * d, seq_row(&c, item, j, g, 0), sizeof(uint16_t) * d);
            memcpy(v_out + (j * hkv + g) * d, seq_row(&c, item, j, g, 1), sizeof(uint16_t) * d);
        }
    release(&c);
    return ORACLE_OK;
}

/* Set the OpenMP thread count (n > 0) and return the count in effect. */
int oracle_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
    return omp_get_max_threads();
#else
    (void)n;
    return 1;
#endif
}
