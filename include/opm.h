/* Outer product mean on one MI355X (gfx950).
 *
 * The operator of Fold-CP Section 3.5 (the equation for z_ijcd): the pair
 * feature of tokens (i, j) is the mean over MSA sequences of the outer
 * product of the projected MSA features a_si and b_sj (each D channels),
 * flattened to D * D values (index c * D + d) and linearly projected to c_z
 * channels.  With the MSA mask m_si (1: token i present in sequence s):
 *
 *     n_ij   = sum_s m_si m_sj
 *     out_ij = W_o vec( (1 / n_ij) sum_s m_si m_sj a_si (x) b_sj ) + b_o
 *
 * (the mean term is 0 where n_ij = 0, so such pairs get b_o).  With every
 * token present, n_ij = |S|, the paper's normalisation.
 *
 * The paper distributes this op as a Cannon-style 2-D ring of partial outer
 * products (Section 3.5: each of sqrt(P) steps adds the products of the
 * sequences the step brings in, and one all-reduce finishes the count).
 * opm_block_accumulate is one device's step of that ring on its pair tile:
 * it adds one panel of sequences into a caller-owned accumulator (sums and
 * counts) and, on the last panel, projects the tile.  opm_forward is the
 * whole op on one GPU (one tile, one panel).
 *
 * Conventions (shared with tri_mul.h): device pointers, status codes
 * TRI_MUL_*, message in tri_mul_last_error(), asynchronous on `stream`
 * (a hipStream_t, NULL = default stream), validation before any launch.
 * Supported: D = 32, c_z = 128.
 */
#ifndef OPM_H
#define OPM_H

#include <stddef.h>
#include <stdint.h>

#include "tri_mul.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct opm_handle_s* opm_handle_t;

typedef struct {
    int32_t d;           /* channels of a and b (D); 32 supported                       */
    int32_t c_z;         /* output channels; 128 supported                              */
    int32_t out_dtype;   /* TRI_MUL_F32 or TRI_MUL_BF16                                 */
    const void* w_o;     /* [c_z][d * d] bf16, flatten index c * d + d' (device)        */
    const void* b_o;     /* [c_z] bf16 (device), or NULL for a zero bias                */
} opm_params_t;

/* One device's step: the pair tile i in [row0, row0 + rows), j in
 * [col0, col0 + cols) and the sequences s in [s0, s0 + slen) of the full
 * tensors (n_total tokens, s_total sequences).  k_index = 0 overwrites the
 * accumulator, later steps add to it; k_index = k_count - 1 also writes the
 * projected tile. */
typedef struct {
    int64_t n_total, s_total;
    int64_t row0, rows, col0, cols;
    int64_t s0, slen;
    int32_t k_index, k_count;
} opm_block_view_t;

/* Copies and repacks w_o, b_o (the caller may free them once `stream`
 * syncs).  EUNSUPPORTED for d != 32 or c_z != 128. */
int opm_init(opm_handle_t* h, const opm_params_t* p, void* stream);

/* Frees the handle (after a device sync); NULL is a no-op. */
int opm_destroy(opm_handle_t h);

/* Bytes of the caller-owned fp32 accumulator of a rows x cols tile: the
 * outer-product sums [rows * d][cols * d] followed by the pair counts
 * [rows][32 * ceil(cols / 32)].  Its contents are private to the library
 * between the steps of one tile. */
int opm_accumulator_size(opm_handle_t h, int64_t rows, int64_t cols, size_t* bytes);

/* Bytes of the per-call workspace of opm_block_accumulate (the step's
 * operands in the contraction's blocked layout: those of the sums
 * transposed, slen rows of tokens * 32 columns each, those of the pair
 * counts plain). */
int opm_workspace_size(opm_handle_t h, int64_t rows, int64_t cols, int64_t slen, size_t* bytes);

/* One step (see opm_block_view_t).  a, b: [s_total][n_total][d] bf16, the
 * projected MSA features (Section 3.5's a and b), read at the view's tokens
 * and sequences; mask: [s_total][n_total] uint8 (nonzero: present), or NULL
 * (all present); acc: accumulator of opm_accumulator_size bytes (16-byte
 * aligned); out_tile: [rows][cols][c_z] of out_dtype, written on the last
 * step only (may be NULL before it); ws: opm_workspace_size bytes, 256-byte
 * aligned.  Rows, cols <= 2048, slen <= 65536.  Errors: EINVAL for null or
 * misaligned pointers, an empty or out-of-range view or bad step indices;
 * ENOMEM for a small workspace; EHIP for a failed launch. */
int opm_block_accumulate(opm_handle_t h, const opm_block_view_t* v, const void* a, const void* b,
                         const uint8_t* mask, float* acc, void* out_tile, void* ws, size_t ws_bytes,
                         void* stream);

/* Bytes of the workspace of opm_forward for S sequences and N tokens (the
 * accumulator plus one step's workspace). */
int opm_forward_workspace_size(opm_handle_t h, int64_t S, int64_t N, size_t* bytes);

/* The whole op on one GPU: out [N][N][c_z] from a, b [S][N][d] and mask
 * [S][N] (or NULL).  N <= 2048, S <= 65536. */
int opm_forward(opm_handle_t h, const void* a, const void* b, const uint8_t* mask, int64_t S, int64_t N,
                void* out, void* ws, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* OPM_H */
