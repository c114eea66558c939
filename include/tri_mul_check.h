/*
 * tri_mul_check.h -- host-side check of the contraction kernel's memory
 * accesses, exported by libtrimul.so next to the operations.
 *
 * The per-channel contraction (Fold-CP, Section 3.3, Eq. 2 / Eq. 3) streams
 * its two operands into LDS with buffer loads whose descriptors and offsets
 * come from a small set of addressing functions.  This call runs those same
 * functions on the host, without a GPU, for one launch shape, and reports
 * whether every load stays inside its operand's allocation and every element
 * a tile needs comes from the address the operand's layout assigns to it.
 * Tests call it for every launch mode of the library before any kernel runs.
 */
#ifndef TRI_MUL_CHECK_H
#define TRI_MUL_CHECK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Operand layouts of the contraction. */
#define TRI_MUL_OPERAND_BLOCKED    0  /* the library's blocked panel (tri_mul_panel_size)          */
#define TRI_MUL_OPERAND_ROW_MAJOR  1  /* [batch][rows][ld] bf16, channel stride `stride` elements  */
#define TRI_MUL_OPERAND_TRANSPOSED 2  /* the operand given as X[k][row] in the blocked panel layout
                                         of K rows (the backward's dC B and dC^T A products)       */

typedef struct {
    int64_t tiles;      /* output tiles of the launch                                  */
    int64_t loads;      /* 64-lane loads visited                                       */
    int64_t elems;      /* needed operand elements visited                             */
    int64_t bad_tiles;  /* tiles taken by no work-group round, or by several          */
    int64_t bad_desc;   /* loads whose buffer descriptor reaches outside the operand  */
    int64_t bad_elem;   /* needed elements read from a wrong address or not at all    */
} tri_mul_load_check_t;

/*
 * Walk the loads of one contraction launch C[b] = A[b] B[b]^T, b < batch,
 * A with M rows, B with N rows, both over K, on a persistent grid of `grid`
 * work-groups.  a_mode / b_mode: TRI_MUL_OPERAND_*; lda, ldb, a_stride,
 * b_stride are used by the row-major layout only (elements; ld a multiple of
 * 8).  a_bytes / b_bytes: the allocation sizes the loads must stay inside.
 * all_channels = 0 visits the first and the last channel (addresses differ
 * between channels only by the channel offset), 1 every channel.
 * Host only; allocates host memory for the tile census; no GPU needed.
 * Returns TRI_MUL_OK with *out filled (violations are reported in the counts,
 * not as an error), or TRI_MUL_EINVAL for null `out`, sizes < 1, a bad mode,
 * a row-major ld below K or not a multiple of 8, or sizes beyond 65536.
 */
int tri_mul_check_contract_loads(int a_mode, int b_mode, int64_t M, int64_t N, int64_t K, int64_t lda,
                                 int64_t ldb, int64_t a_stride, int64_t b_stride, int batch, uint64_t a_bytes,
                                 uint64_t b_bytes, int grid, int all_channels, tri_mul_load_check_t* out);

/*
 * The same walk over the contraction kernel's accesses to its result C in
 * the pair-blocked result layout (tri_mul_contract): M rows, N columns,
 * `batch` channels, element (b, i, j) at ((i * J + j / 32) * batch + b) * 32
 * + j % 32 floats with J = ceil(N / 32), c_bytes allocated.  Each MFMA wave
 * reads (when accumulating) and writes its 64 x 128 part of a tile through
 * one buffer descriptor per 32-column block.  Reports in *out: tiles, the
 * 64-lane register groups visited (loads), the elements with row < M and
 * column < N visited (elems), descriptors reaching outside c_bytes
 * (bad_desc), and accesses at an address other than the layout's, inside
 * the descriptor but outside C's rows or column blocks, or elements
 * accessed never or more than once (bad_elem); bad_tiles is 0.
 * all_channels as above.  Host only.  Returns TRI_MUL_OK, or
 * TRI_MUL_EINVAL for null `out` or sizes outside [1, 65536].
 */
int tri_mul_check_contract_result(int64_t M, int64_t N, int batch, uint64_t c_bytes, int all_channels,
                                  tri_mul_load_check_t* out);

#ifdef __cplusplus
}
#endif

#endif /* TRI_MUL_CHECK_H */
