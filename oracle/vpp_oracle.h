/*
 * vpp_oracle.h -- plain fp64 CPU reference for chunked-prefill causal attention.
 *
 * TEST INFRASTRUCTURE ONLY. This library is the checker, not the product. Only
 * tests/, __graft_entry__.smoke() and the cpu_baseline leg of bench.py may load
 * or call it. It shares no code, header, table or helper with the HIP library.
 *
 * What it computes: Eq. (1) of the paper (section 2.1, "Transformer
 * Architecture"), softmax(Q K^T / sqrt(d)) V, with the causal rule stated right
 * after it (a token sees itself and the tokens before it), applied to the
 * chunked prefill of section 2.4: the queries of one chunk sit at in-request
 * positions prefix_len .. prefix_len + len - 1 and see every key of their own
 * request up to and including their own position (the cached prefix plus the
 * chunk itself).
 */
#ifndef VPP_ORACLE_H
#define VPP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define VPP_ORACLE_OK 0
#define VPP_ORACLE_EINVAL (-1)    /* an argument is out of range            */
#define VPP_ORACLE_ENOMEM (-2)    /* host allocation failed                 */
#define VPP_ORACLE_ESELFCHECK (-3) /* softmax weights did not sum to 1      */

/*
 * Evaluate selected (query row, query head) items in fp64.
 *
 * Tensors hold bf16 values as raw 16-bit patterns, on the host, indexed as
 *   q[t*q_st + h*q_sh + c]   t = chunk-local token, h = query head, c < dqk
 *   k[T*k_st + g*k_sh + c]   T = cache row, g = kv head, c < dqk
 *   v[T*v_st + g*v_sh + c]   c < dv
 * Strides are in elements. Query head h reads kv head g = h / (hq / hkv)
 * (contiguous groups).
 *
 * Segments: chunk rows cu_q[s] .. cu_q[s+1]-1 belong to segment s. Row r of
 * segment s has in-request position i = prefix_len[s] + (r - cu_q[s]) and sees
 * cache rows kv_start[s] + j for j = 0 .. i.
 *
 * Items: item n is (row item_row[n], query head item_head[n]); its result goes
 * to out[n*dv + c] and lse[n] (natural logarithm of the softmax denominator,
 * including the scale). scale is used as given.
 *
 * n_threads <= 0 uses every online core. Returns VPP_ORACLE_OK or a negative
 * code above; on error the outputs are unspecified.
 */
int vpp_oracle_attn(const uint16_t* q, int64_t q_st, int64_t q_sh,
                    const uint16_t* k, int64_t k_st, int64_t k_sh,
                    const uint16_t* v, int64_t v_st, int64_t v_sh,
                    int32_t hq, int32_t hkv, int32_t dqk, int32_t dv,
                    double scale,
                    int32_t n_seg, const int32_t* cu_q,
                    const int64_t* kv_start, const int64_t* prefix_len,
                    int64_t n_items, const int64_t* item_row,
                    const int32_t* item_head,
                    double* out, double* lse, int32_t n_threads);

/* Number of threads vpp_oracle_attn would use for n_threads <= 0. */
int32_t vpp_oracle_default_threads(void);

#ifdef __cplusplus
}
#endif
#endif /* VPP_ORACLE_H */
