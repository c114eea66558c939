/* Triangle attention core on one MI355X (gfx950).
 *
 * Fold-CP Section 3.2, Eq. 1 (attention around the starting node): for row
 * i of the pair representation, head h and query pair (i, j),
 *
 *     out_ijh = sum_k softmax_k( q_ijh . k_ikh / sqrt(32) + b_hjk ) v_ikh
 *
 * over the keys k with mask[k] != 0 (Eq. 1's mask_bias; if no key is
 * present the output is 0).  q, k, v are Eq. 1's projections of z and b its
 * tri_bias(z), which does not depend on i.  The paper runs the keys around a
 * ring in chunks and merges the partial results with a running log-sum-exp;
 * tri_attn_chunk is one such step (it merges keys [k0, k0 + klen) into a
 * caller-owned state), tri_attn_forward the whole op in one call.
 *
 * Layouts (device pointers, bf16 unless stated): q, k, v [rows][n][heads][32]
 * (head dimension 32); bias [heads][n][ld_bias] (ld_bias % 8 == 0,
 * ld_bias >= n); mask uint8 [n] or NULL (all present); out
 * [rows][n][heads][32] of out_dtype (TRI_MUL_F32 or TRI_MUL_BF16).
 * Precision: with fp32 output the softmax weights enter the weighted sum
 * of v with ~16 mantissa bits; with bf16 output with 8 (bf16), an error of
 * the same order as the output's own rounding.
 * Status codes and the error message as in tri_mul.h; asynchronous on
 * `stream` (hipStream_t, NULL = default); validation before any launch.
 */
#ifndef TRIATTN_H
#define TRIATTN_H

#include <stddef.h>
#include <stdint.h>

#include "tri_mul.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int64_t rows;       /* rows i (independent attentions of n queries over n keys)      */
    int64_t n;          /* tokens per row: queries and keys                               */
    int32_t heads;      /* 1 .. 16                                                        */
    int32_t out_dtype;  /* TRI_MUL_F32 or TRI_MUL_BF16                                    */
    int64_t ld_bias;    /* row stride of bias (elements)                                  */
    int64_t k0, klen;   /* this step's keys [k0, k0 + klen); k0 % 8 == 0                  */
    int32_t k_index;    /* 0: start a fresh state; > 0: merge into the state             */
    int32_t k_count;    /* k_index == k_count - 1 writes out (and not the state)          */
} tri_attn_view_t;

/* Bytes of the fp32 state of one chunked attention: the unnormalised
 * outputs [rows][n][heads][32], then the running maxima and sums
 * [rows][heads][n] each.  Private to the library between the steps. */
int tri_attn_state_size(const tri_attn_view_t* v, size_t* bytes);

/* One step: merges keys [k0, k0 + klen) into `state` (16-byte aligned;
 * read unless k_index == 0); on the last step writes out instead of the
 * state.  Steps of one attention must cover disjoint key ranges.  Errors:
 * EINVAL for null or misaligned pointers, bad sizes or step indices. */
int tri_attn_chunk(const tri_attn_view_t* v, const void* q, const void* k, const void* vv, const void* bias,
                   const uint8_t* mask, float* state, void* out, void* stream);

/* The whole op in one call (all n keys, no state). */
int tri_attn_forward(const void* q, const void* k, const void* v, const void* bias, const uint8_t* mask,
                     int64_t rows, int64_t n, int32_t heads, int64_t ld_bias, int32_t out_dtype, void* out,
                     void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TRIATTN_H */
