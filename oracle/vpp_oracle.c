/*
 * vpp_oracle.c -- plain fp64 CPU reference for chunked-prefill causal attention.
 *
 * TEST INFRASTRUCTURE ONLY: the checker, not the product. Only tests/,
 * __graft_entry__.smoke() and the cpu_baseline leg of bench.py may load it.
 * It shares nothing with the HIP library.
 *
 * It is the plain definition, written out once per checked item, with no
 * blocking or reordering: Eq. (1) of the paper (section 2.1), softmax of the
 * scaled dot products followed by the weighted sum of values, restricted by the
 * causal rule of section 2.1 to keys at positions 0..i of the query's own
 * request, where i is the query's in-request position. Section 2.4 gives the
 * chunk semantics: a later chunk's queries see the whole cached prefix plus
 * the earlier tokens of their own chunk.
 *
 * Arithmetic: inputs are bf16 bit patterns, widened exactly to double; every
 * product, sum, exp and log is done in double in natural key order. The
 * maximum score is subtracted before exponentiation so that no term
 * overflows; this leaves the quotient unchanged.
 */
#define _GNU_SOURCE
#include "vpp_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

/* bf16 is the upper half of an IEEE binary32: shift the bits up, reinterpret
 * as float, then widen to double (both steps are exact). */
static double bf16_to_double(uint16_t bits) {
    uint32_t w = ((uint32_t)bits) << 16;
    float f;
    memcpy(&f, &w, sizeof f);
    return (double)f;
}

typedef struct {
    const uint16_t *q, *k, *v;
    int64_t q_st, q_sh, k_st, k_sh, v_st, v_sh;
    int32_t hq, hkv, dqk, dv;
    double scale;
    int32_t n_seg;
    const int32_t* cu_q;
    const int64_t *kv_start, *prefix_len;
    int64_t n_items;
    const int64_t* item_row;
    const int32_t* item_head;
    double *out, *lse;
    int64_t max_keys;
    /* shared work counter and first error seen */
    int64_t next;
    int status;
    pthread_mutex_t mu;
} job_t;

/* Segment that owns chunk row r: the s with cu_q[s] <= r < cu_q[s+1]. */
static int32_t find_segment(const int32_t* cu_q, int32_t n_seg, int64_t r) {
    int32_t lo = 0, hi = n_seg - 1;
    while (lo < hi) {
        int32_t mid = (lo + hi + 1) / 2;
        if ((int64_t)cu_q[mid] <= r) lo = mid; else hi = mid - 1;
    }
    return lo;
}

/* One (row, head) item: the definition, step by step. */
static int one_item(const job_t* J, int64_t n, double* s, double* acc) {
    const int64_t r = J->item_row[n];
    const int32_t h = J->item_head[n];
    const int32_t group = J->hq / J->hkv;
    const int32_t g = h / group;
    const int32_t seg = find_segment(J->cu_q, J->n_seg, r);
    /* in-request position of this query and the cache row of its key 0 */
    const int64_t i = J->prefix_len[seg] + (r - J->cu_q[seg]);
    const int64_t base = J->kv_start[seg];
    const uint16_t* qrow = J->q + r * J->q_st + (int64_t)h * J->q_sh;

    /* scores s_j = scale * <q, k_j> for the visible keys j = 0..i */
    double m = -INFINITY;
    for (int64_t j = 0; j <= i; ++j) {
        const uint16_t* krow = J->k + (base + j) * J->k_st + (int64_t)g * J->k_sh;
        double dot = 0.0;
        for (int32_t c = 0; c < J->dqk; ++c)
            dot += bf16_to_double(qrow[c]) * bf16_to_double(krow[c]);
        s[j] = J->scale * dot;
        if (s[j] > m) m = s[j];
    }

    /* softmax numerators and denominator, then the weighted sum of values */
    double l = 0.0;
    for (int32_t c = 0; c < J->dv; ++c) acc[c] = 0.0;
    for (int64_t j = 0; j <= i; ++j) {
        const double e = exp(s[j] - m);
        s[j] = e;
        l += e;
        const uint16_t* vrow = J->v + (base + j) * J->v_st + (int64_t)g * J->v_sh;
        for (int32_t c = 0; c < J->dv; ++c) acc[c] += e * bf16_to_double(vrow[c]);
    }
    for (int32_t c = 0; c < J->dv; ++c) J->out[n * J->dv + c] = acc[c] / l;
    J->lse[n] = m + log(l);

    /* self-check: the softmax weights of the row sum to one */
    double wsum = 0.0;
    for (int64_t j = 0; j <= i; ++j) wsum += s[j] / l;
    if (!(fabs(wsum - 1.0) <= 1e-12)) return VPP_ORACLE_ESELFCHECK;
    return VPP_ORACLE_OK;
}

static void* worker(void* arg) {
    job_t* J = (job_t*)arg;
    double* s = (double*)malloc(sizeof(double) * (size_t)(J->max_keys > 0 ? J->max_keys : 1));
    double* acc = (double*)malloc(sizeof(double) * (size_t)J->dv);
    int st = (s && acc) ? VPP_ORACLE_OK : VPP_ORACLE_ENOMEM;
    for (;;) {
        int64_t n;
        pthread_mutex_lock(&J->mu);
        if (st != VPP_ORACLE_OK && J->status == VPP_ORACLE_OK) J->status = st;
        n = (J->status == VPP_ORACLE_OK) ? J->next++ : J->n_items;
        pthread_mutex_unlock(&J->mu);
        if (n >= J->n_items) break;
        st = one_item(J, n, s, acc);
    }
    free(s);
    free(acc);
    return NULL;
}

int32_t vpp_oracle_default_threads(void) {
    long n = sysconf(_SC_NPROCESSORS_ONLN);
    return (int32_t)(n > 0 ? n : 1);
}

int vpp_oracle_attn(const uint16_t* q, int64_t q_st, int64_t q_sh,
                    const uint16_t* k, int64_t k_st, int64_t k_sh,
                    const uint16_t* v, int64_t v_st, int64_t v_sh,
                    int32_t hq, int32_t hkv, int32_t dqk, int32_t dv,
                    double scale,
                    int32_t n_seg, const int32_t* cu_q,
                    const int64_t* kv_start, const int64_t* prefix_len,
                    int64_t n_items, const int64_t* item_row,
                    const int32_t* item_head,
                    double* out, double* lse, int32_t n_threads) {
    if (!q || !k || !v || !cu_q || !kv_start || !prefix_len || !out || !lse)
        return VPP_ORACLE_EINVAL;
    if (n_items < 0 || (n_items > 0 && (!item_row || !item_head))) return VPP_ORACLE_EINVAL;
    if (hq <= 0 || hkv <= 0 || hq % hkv != 0 || dqk <= 0 || dv <= 0 || n_seg <= 0)
        return VPP_ORACLE_EINVAL;
    if (cu_q[0] != 0) return VPP_ORACLE_EINVAL;
    for (int32_t s = 0; s < n_seg; ++s) {
        if (cu_q[s + 1] < cu_q[s] || prefix_len[s] < 0 || kv_start[s] < 0)
            return VPP_ORACLE_EINVAL;
    }
    /* longest key list over the requested items sizes the per-thread buffer */
    int64_t max_keys = 0;
    for (int64_t n = 0; n < n_items; ++n) {
        if (item_row[n] < 0 || item_row[n] >= cu_q[n_seg]) return VPP_ORACLE_EINVAL;
        if (item_head[n] < 0 || item_head[n] >= hq) return VPP_ORACLE_EINVAL;
        int32_t seg = find_segment(cu_q, n_seg, item_row[n]);
        int64_t keys = prefix_len[seg] + (item_row[n] - cu_q[seg]) + 1;
        if (keys > max_keys) max_keys = keys;
    }
    if (n_items == 0) return VPP_ORACLE_OK;

    job_t J;
    memset(&J, 0, sizeof J);
    J.q = q; J.k = k; J.v = v;
    J.q_st = q_st; J.q_sh = q_sh; J.k_st = k_st; J.k_sh = k_sh; J.v_st = v_st; J.v_sh = v_sh;
    J.hq = hq; J.hkv = hkv; J.dqk = dqk; J.dv = dv; J.scale = scale;
    J.n_seg = n_seg; J.cu_q = cu_q; J.kv_start = kv_start; J.prefix_len = prefix_len;
    J.n_items = n_items; J.item_row = item_row; J.item_head = item_head;
    J.out = out; J.lse = lse; J.max_keys = max_keys;
    J.next = 0; J.status = VPP_ORACLE_OK;
    pthread_mutex_init(&J.mu, NULL);

    int32_t nt = n_threads > 0 ? n_threads : vpp_oracle_default_threads();
    if (nt > n_items) nt = (int32_t)n_items;
    pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nt);
    if (!th) { pthread_mutex_destroy(&J.mu); return VPP_ORACLE_ENOMEM; }
    int32_t started = 0;
    for (int32_t t = 1; t < nt; ++t) {
        if (pthread_create(&th[t], NULL, worker, &J) != 0) break;
        started = t;
    }
    worker(&J); /* the calling thread works too */
    for (int32_t t = 1; t <= started; ++t) pthread_join(th[t], NULL);
    free(th);
    pthread_mutex_destroy(&J.mu);
    return J.status;
}
