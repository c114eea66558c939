/*
 * tri_mul.h -- C ABI of the MI355X (gfx950) triangular multiplicative update.
 *
 * The operation (Fold-CP, Section 3.3, Eq. 2 outgoing and Eq. 3 incoming):
 *
 *   outgoing:  C[i][j][c] = sum_k a[i][k][c] * b[j][k][c]
 *   incoming:  C[i][j][c] = sum_k a[k][i][c] * b[k][j][c]
 *
 * where a and b are gated linear maps of the pair tensor z
 * (Section 3.3 names the projections and their element-wise gate without
 * spelling out the layer; the layer below is the usual one).  For every
 * pair (i, j), with pair mask m_ij = m_i * m_j:
 *
 *   x_ij   = LN_in(z_ij)                              over c_z channels
 *   a_ij   = m_ij * sigmoid(W_ga x_ij) * (W_a x_ij)   c channels
 *   b_ij   = m_ij * sigmoid(W_gb x_ij) * (W_b x_ij)
 *   out_ij = m_ij * sigmoid(W_g x_ij) * (W_o LN_out(C_ij))   c_z channels
 *
 * LN is LayerNorm with the biased variance and epsilon ln_eps.  The library
 * returns the update out (the right-hand side of Eq. 2/3); the residual add
 * z + out is the caller's.  Padded tokens (mask 0) contribute exactly zero to
 * every sum and get exactly zero output.
 *
 * The paper shards z over a sqrt(P) x sqrt(P) grid (Section 2.1.1) and runs
 * the contraction as a Cannon ring in which every step multiplies the resident
 * row block of a with the column block of b and adds the product into the
 * output block (Section 3.3, Fig. 2b).  tri_mul_block_accumulate() is one such
 * step for one device's tile.
 *
 * Conventions for every call:
 *   - Every tensor pointer is a DEVICE pointer (hipMalloc / torch CUDA
 *     memory) unless stated otherwise; every struct pointer is a HOST pointer.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Work is enqueued asynchronously on it; device faults surface at the
 *     caller's next synchronisation.
 *   - Arguments are validated synchronously before anything is enqueued.
 *     On failure nothing is launched and a negative status is returned;
 *     tri_mul_last_error() then describes the failure (thread-local text).
 *   - No C++ exception crosses this interface.
 *   - One handle may be used from one stream at a time.
 *   - Tensor pointers must be 16-byte aligned; row strides given in elements
 *     must keep every row 16-byte aligned.
 *   - Supported sizes: c_z = c = 128.  1 <= N <= 65536 (and N*N*c fits in
 *     int64).
 */
#ifndef TRI_MUL_H
#define TRI_MUL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define TRI_MUL_OK            0
#define TRI_MUL_EINVAL       -1  /* null pointer, bad size, bad alignment, bad enum */
#define TRI_MUL_EUNSUPPORTED -2  /* valid but unsupported configuration           */
#define TRI_MUL_ENOMEM       -3  /* workspace too small or device allocation failed */
#define TRI_MUL_EHIP         -4  /* the HIP runtime reported an error             */

/* Storage types. */
#define TRI_MUL_F32  0           /* float32 storage, float32 arithmetic           */
#define TRI_MUL_BF16 1           /* bfloat16 storage, float32 accumulation        */

/* Directions (Eq. 2 and Eq. 3). */
#define TRI_MUL_OUTGOING 0
#define TRI_MUL_INCOMING 1

typedef struct tri_mul_handle_s* tri_mul_handle_t;

/* Layer parameters.  All weight pointers are DEVICE pointers of type `dtype`,
 * linear maps in [out][in] row-major layout (y = W x):
 *   ln_in_w, ln_in_b   [c_z]        input LayerNorm gain and bias
 *   w_a, w_ga          [c][c_z]     value / gate projection of a
 *   w_b, w_gb          [c][c_z]     value / gate projection of b
 *   w_g                [c_z][c_z]   output gate projection
 *   ln_out_w, ln_out_b [c]          output LayerNorm gain and bias
 *   w_o                [c_z][c]     output projection
 * The library copies (and repacks) them during tri_mul_init; the caller may
 * free its copies once tri_mul_init has returned. */
typedef struct {
    int32_t c_z;
    int32_t c;
    int32_t dtype;       /* TRI_MUL_F32 or TRI_MUL_BF16: z, weights, panels */
    int32_t out_dtype;   /* TRI_MUL_F32 or TRI_MUL_BF16: out               */
    float   ln_eps;      /* LayerNorm epsilon, e.g. 1e-5                    */
    const void* ln_in_w;
    const void* ln_in_b;
    const void* w_a;
    const void* w_ga;
    const void* w_b;
    const void* w_gb;
    const void* w_g;
    const void* ln_out_w;
    const void* ln_out_b;
    const void* w_o;
} tri_mul_params_t;

/* One device's tile of the 2-D pair grid and one k-panel of the ring
 * (Section 2.1.1 tiling; Section 3.3 ring step).  Token indices are global:
 *   output rows  i in [row0, row0 + rows),  columns j in [col0, col0 + cols),
 *   k-panel      k in [k0, k0 + klen) of n_total tokens.
 * ld_a / ld_b are the row strides (elements) of the a / b panels, >= klen,
 * multiples of 8, at most 65536 (larger strides return TRI_MUL_EUNSUPPORTED:
 * the kernels address a panel tile with 32-bit byte offsets).  k_index / k_count number the panels of one tile: the call
 * with k_index == 0 overwrites the accumulator, later calls add to it, and
 * the call with k_index == k_count - 1 also runs the epilogue. */
typedef struct {
    int64_t n_total;
    int64_t row0, col0;
    int64_t rows, cols;
    int64_t k0, klen;
    int64_t ld_a, ld_b;
    int32_t k_index, k_count;
} tri_mul_block_view_t;

/* Create a handle: validates `p`, allocates device buffers for the repacked
 * weights and copies them (synchronously with respect to `stream`).
 * Returns TRI_MUL_EUNSUPPORTED unless c_z == c == 128, and (bf16 storage)
 * when a projection weight matrix or the input LayerNorm's gain and bias are
 * so large that the projection's fp16 matrix-core operands would overflow
 * even scaled by 2^-40 (a largest |W| entry, or sqrt(c_z - 1) max|gamma| +
 * max|beta|, above about 6.5e4 * 2^40). */
int tri_mul_init(tri_mul_handle_t* h, const tri_mul_params_t* p, void* stream);

/* Free the handle's device buffers (after the device has finished with
 * them).  Destroying NULL is a no-op returning TRI_MUL_OK. */
int tri_mul_destroy(tri_mul_handle_t h);

/* Text of the last failure on the calling thread ("" if none). */
const char* tri_mul_last_error(void);

/* Bytes of device workspace tri_mul_outgoing / tri_mul_incoming need for N
 * tokens: the two contraction operands (panel layout, see tri_mul_project)
 * and the fp32 contraction result (result layout, see tri_mul_contract), each
 * 256-byte aligned.  *bytes is a HOST pointer.  With bf16 storage the full
 * calls keep the operands transposed there -- the panels tri_mul_project
 * writes for the opposite direction, contracted by
 * tri_mul_contract_transposed; with fp32 storage the direction's own. */
int tri_mul_workspace_size(tri_mul_handle_t h, int64_t N, size_t* bytes);

/* The full update, Eq. 2 (outgoing) / Eq. 3 (incoming).
 *   z     [N][N][c_z]  dtype, row-major pair tensor
 *   mask  [N]          uint8 token mask (nonzero = real token); NULL = all real
 *   out   [N][N][c_z]  out_dtype; receives the update; must not alias z or ws
 *   ws    workspace of >= tri_mul_workspace_size(N) bytes, 256-byte aligned
 * Returns TRI_MUL_ENOMEM if ws_bytes is too small. */
int tri_mul_outgoing(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N,
                     void* out, void* ws, size_t ws_bytes, void* stream);
int tri_mul_incoming(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N,
                     void* out, void* ws, size_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, hosts that forbid hipMalloc): the full update
 * of tri_mul_outgoing (direction TRI_MUL_OUTGOING) or tri_mul_incoming
 * (TRI_MUL_INCOMING), with the same z, mask, N, out and stream arguments and
 * the same results, but no workspace argument.  The workspace lives in a
 * fixed device scratch array of 256 MiB (268435456 bytes) that every GPU the
 * library runs on holds until the process ends; the call itself allocates
 * nothing (no hipMalloc, hipFree or allocating library routine).
 *   - N is limited to sizes whose tri_mul_workspace_size fits the scratch
 *     (bf16 storage: N <= 512); larger N returns TRI_MUL_EUNSUPPORTED.
 *   - Every call on one GPU shares that GPU's scratch, which keeps the last
 *     call's contents: calls that overlap in time on one GPU (different
 *     streams, threads or handles) race and corrupt each other's results.
 *     Serialise them (one stream, or events between streams).
 *   - The scratch needs no clearing: every element a call reads was written
 *     earlier in the same call.
 * Errors: those of tri_mul_outgoing, plus TRI_MUL_EINVAL for a bad direction. */
int tri_mul_update_noalloc(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N,
                           int32_t direction, void* out, void* stream);

/* One ring step of one device tile (Section 3.3, Fig. 2b):
 *   acc (+)= A_c * diag(m_k) * B_c^T   for every hidden channel c
 *   a_panel  [c][rows][ld_a]  dtype, a_panel[c][i][k] = a at (row0+i, k0+k)
 *   b_panel  [c][cols][ld_b]  dtype, b_panel[c][j][k] = b at (col0+j, k0+k)
 *   acc      [c][rows][cols]  float32, caller-owned, overwritten when
 *            k_index == 0 and accumulated into otherwise
 *   mask     [n_total] uint8 token mask (NULL = all real): column k counts only
 *            if mask[k0+k] != 0; rows/cols use mask[row0+i] * mask[col0+j]
 *   z_tile   [rows][cols][c_z] dtype (read only when k_index == k_count-1):
 *            the pair tensor of the tile, source of the output gate
 *   out_tile [rows][cols][c_z] out_dtype (written only when k_index ==
 *            k_count-1): the update of the tile
 * The panels are direction-agnostic (for the incoming update the caller
 * supplies the transposed operands). */
int tri_mul_block_accumulate(tri_mul_handle_t h, const tri_mul_block_view_t* v,
                             const void* a_panel, const void* b_panel, float* acc,
                             const uint8_t* mask, const void* z_tile, void* out_tile,
                             void* stream);

/* Bytes of device workspace tri_mul_block_accumulate_ws and
 * tri_mul_block_repack need for the view's sizes (rows, cols, klen): both
 * panels repacked, masked, into the blocked operand layout (see
 * tri_mul_project), 128 * ceil(rows/256) * ceil(klen/32) * 16 KB + the same
 * for cols, and the staged k-mask (ceil(klen/32) * 32 bytes), each part
 * 256-byte aligned; 0 for the fp32 path.  *bytes is a HOST pointer. */
int tri_mul_block_workspace_size(tri_mul_handle_t h, const tri_mul_block_view_t* v, size_t* bytes);

/* The same ring step as tri_mul_block_accumulate (same arguments, results
 * and errors) through a caller-owned workspace (256-byte aligned, at least
 * tri_mul_block_workspace_size bytes, else TRI_MUL_ENOMEM): the two panels
 * are first repacked, with the mask applied, into the blocked layout, so
 * the contraction reads whole 16 KB blocks instead of 64-byte row pieces.
 * The workspace is scratch for the duration of the call (stream-ordered). */
int tri_mul_block_accumulate_ws(tri_mul_handle_t h, const tri_mul_block_view_t* v,
                                const void* a_panel, const void* b_panel, float* acc,
                                const uint8_t* mask, const void* z_tile, void* out_tile,
                                void* ws, size_t ws_bytes, void* stream);

/* The ring step of tri_mul_block_accumulate_ws split in two, with the
 * accumulator in the pair-blocked result layout, so that a caller can
 * repack the next k-panel on a second stream while the current one is
 * contracted (Section 3.3, Fig. 2b: each ring step adds one panel product
 * into the output block; the repack of panel p + 1 has no dependence on
 * the product of panel p).  bf16 storage path only (else
 * TRI_MUL_EUNSUPPORTED).
 *
 * tri_mul_block_accumulator_size: bytes of the packed accumulator for the
 *   view's rows and cols: element (hidden channel c, tile row i, tile
 *   column j) at ((i * J + j / 32) * 128 + c) * 32 + j % 32 floats, J =
 *   ceil(cols / 32) (the result layout of tri_mul_contract); rows * J * 32 *
 *   128 * 4 bytes.  *bytes is a HOST pointer.
 * tri_mul_block_repack: repacks a_panel and b_panel (the arguments of
 *   tri_mul_block_accumulate), with the k-range of mask applied, into ws
 *   (tri_mul_block_workspace_size bytes, 256-byte aligned; TRI_MUL_ENOMEM if
 *   smaller).  Only the view's sizes, k0 and strides are used.
 * tri_mul_block_accumulate_packed: acc (+)= the product of the panels
 *   repacked in ws by tri_mul_block_repack for the same view (overwritten
 *   when k_index == 0, accumulated into otherwise); when k_index ==
 *   k_count - 1 also the epilogue into out_tile, as tri_mul_block_accumulate.
 *   reserve_cus compute units (0 .. CUs - 8) are left to concurrent work,
 *   e.g. the next panel's repack on another stream (the contraction runs on
 *   the rest, rounded down to a multiple of 8).  acc is 16-byte aligned.
 * The caller orders the calls with events: the repack of a panel before its
 * accumulate, and a workspace reused only after the accumulate that read it
 * has finished.  tri_mul_block_repack touches no device buffer of the handle
 * (its staged k-mask lives in ws), so it may run on a second stream while
 * other calls of the same handle run on the first -- the one exception to
 * the one-stream-per-handle rule.  Results equal tri_mul_block_accumulate's up to the order
 * of the fp32 additions over k-panels (identical per panel). */
int tri_mul_block_accumulator_size(tri_mul_handle_t h, const tri_mul_block_view_t* v, size_t* bytes);
int tri_mul_block_repack(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* a_panel,
                         const void* b_panel, const uint8_t* mask, void* ws, size_t ws_bytes, void* stream);
int tri_mul_block_accumulate_packed(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* ws,
                                    size_t ws_bytes, float* acc, const uint8_t* mask, const void* z_tile,
                                    void* out_tile, int32_t reserve_cus, void* stream);

/* The ring with the panels travelling in the contraction's blocked operand
 * layout (Section 3.3, Fig. 2b).  Each device projects its own tile of z
 * once per layer; the panels it passes round the ring are those projections,
 * so writing them in the layout the contraction reads removes the repack
 * from every ring step.  bf16 storage path only (else TRI_MUL_EUNSUPPORTED).
 *
 * Blocked panel of m rows and klen contraction indices: for hidden channel c,
 *   element (c, i, k) at ((c * T + i / 256) * S + k / 32) * 8192 + (i % 256) * 32 + k % 32
 * with T = ceil(m / 256), S = ceil(klen / 32) (the operand layout of
 * tri_mul_project for a rectangle); entries with i >= m hold unspecified
 * values and never contribute, entries with k >= klen are zero.
 *
 * tri_mul_block_panel_size: bytes of a blocked panel of m = rows rows and
 *   klen contraction indices, 128 * T * S * 16 KB.  *bytes is a HOST pointer.
 *   rows, klen <= 65536.
 * tri_mul_block_project: the tile's input LayerNorm, gated projections and
 *   pair mask (as tri_mul_project) written as two blocked panels.
 *     z_tile   [rows][ld_z][c_z] dtype: pair (row0 + i, col0 + j) at
 *              z_tile[i][j], ld_z >= cols (at most 65536)
 *     mask     [n_total] uint8 token mask (NULL = all real); a(p, q) and
 *              b(p, q) are 0 unless mask[p] and mask[q] are both nonzero
 *   direction TRI_MUL_OUTGOING: a_panel[c][i][k] = a at (row0 + i, col0 + k),
 *     m = rows, klen = cols: the a-panel of k-range [col0, col0 + cols) for
 *     output rows [row0, row0 + rows), and likewise b the b-panel for output
 *     columns [row0, row0 + rows) (Eq. 2 contracts the second token index).
 *   direction TRI_MUL_INCOMING: a_panel[c][i][k] = a at (row0 + k, col0 + i),
 *     m = cols, klen = rows: the a-panel of k-range [row0, row0 + rows) for
 *     output rows [col0, col0 + cols), and likewise b the b-panel for output
 *     columns [col0, col0 + cols) (Eq. 3 contracts the first token index).
 *   a_panel, b_panel: tri_mul_block_panel_size(m, klen) bytes each, 16-byte
 *   aligned.  Uses the handle's staging buffer: one stream per handle.
 * tri_mul_block_accumulate_blocked: the ring step of
 *   tri_mul_block_accumulate_packed with the two panels given directly in the
 *   blocked layout (a_panel: m = rows, b_panel: m = cols, both klen; the mask
 *   was applied when they were projected, so mask serves only the epilogue);
 *   ld_a and ld_b of the view are not used.  acc is the packed accumulator
 *   of tri_mul_block_accumulator_size (overwritten when k_index == 0,
 *   accumulated into otherwise); the call with k_index == k_count - 1 also
 *   runs the epilogue into out_tile.  reserve_cus as for
 *   tri_mul_block_accumulate_packed.  Given the panels that
 *   tri_mul_block_repack writes for the same values, the results are
 *   identical to tri_mul_block_accumulate_packed's.
 * tri_mul_block_accumulate_transposed: the same ring step from the two
 *   panels transposed -- at_panel holds A^T (m = klen rows, rows
 *   contraction indices), bt_panel B^T (m = klen, cols), i.e. what
 *   tri_mul_block_project writes from the same z tiles with the OPPOSITE
 *   direction; other arguments, accumulator, epilogue and errors as
 *   tri_mul_block_accumulate_blocked, and the sums are bitwise the same.
 *   On gfx950 this operand order is the faster one (as for the full
 *   update, see tri_mul_contract_transposed). */
int tri_mul_block_panel_size(tri_mul_handle_t h, int64_t rows, int64_t klen, size_t* bytes);
int tri_mul_block_project(tri_mul_handle_t h, const void* z_tile, int64_t ld_z, const uint8_t* mask, int64_t n_total,
                          int64_t row0, int64_t col0, int64_t rows, int64_t cols, int32_t direction, void* a_panel,
                          void* b_panel, void* stream);
int tri_mul_block_accumulate_blocked(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* a_panel,
                                     const void* b_panel, float* acc, const uint8_t* mask, const void* z_tile,
                                     void* out_tile, int32_t reserve_cus, void* stream);
int tri_mul_block_accumulate_transposed(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* at_panel,
                                        const void* bt_panel, float* acc, const uint8_t* mask, const void* z_tile,
                                        void* out_tile, int32_t reserve_cus, void* stream);

/* The three stages of tri_mul_outgoing / tri_mul_incoming, exposed so that
 * callers can time or check them one by one.
 *
 * Operand ("panel") layout.  The contraction operands A, B hold, for every
 * hidden channel c, an N x N matrix X_c[i][k] in 256 x 32 blocks: element
 * (c, i, k) is at index
 *     ((c * T + i / 256) * S + k / 32) * 8192 + (i % 256) * 32 + k % 32
 * with T = ceil(N / 256) and S = ceil(N / 32), so one operand takes
 * c * T * 256 * S * 32 elements.  Padding elements (i >= N or k >= N) hold
 * unspecified values and never contribute.
 *
 * tri_mul_panel_size: bytes of one operand for N tokens (*bytes is HOST). */
int tri_mul_panel_size(tri_mul_handle_t h, int64_t N, size_t* bytes);

/* tri_mul_project: input LayerNorm, gated projections and pair mask.
 *   Writes A, B (dtype, panel layout, tri_mul_panel_size bytes each):
 *   outgoing X_c[i][k] = a[i][k][c], incoming X_c[i][k] = a[k][i][c]
 *   (likewise B), so that either direction becomes C[c] = A[c] * B[c]^T. */
int tri_mul_project(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N,
                    int32_t direction, void* a_panels, void* b_panels, void* stream);

/* tri_mul_contract: C_c[i][j] = sum_k A_c[i][k] * B_c[j][k] for all c.
 *   A, B in the panel layout above.  C (float32, overwritten) in the result
 *   layout: element (channel ch, i, j) at ((i * J + j / 32) * c + ch) * 32 +
 *   j % 32 with J = ceil(N / 32) -- the c channels of 32 consecutive pairs of
 *   a row are one contiguous block; C takes N * J * 32 * c floats. */
int tri_mul_contract(tri_mul_handle_t h, const void* a_panels, const void* b_panels,
                     int64_t N, float* c_out, void* stream);

/* tri_mul_contract_transposed: the same C from the operands given
 * transposed, AT_c = A_c^T and BT_c = B_c^T in the panel layout:
 * C_c[i][j] = sum_k AT_c[k][i] * BT_c[k][j].  Since the outgoing operands
 * are the incoming ones transposed and vice versa, tri_mul_project with the
 * opposite direction writes exactly AT and BT, and
 *     tri_mul_contract_transposed(project(z, opposite direction))
 * is bitwise equal to tri_mul_contract(project(z, direction)).  On gfx950
 * this order is the faster one (the full calls use it with bf16 storage).
 * bf16 storage only (TRI_MUL_EUNSUPPORTED otherwise); other arguments and
 * errors as tri_mul_contract. */
int tri_mul_contract_transposed(tri_mul_handle_t h, const void* at_panels, const void* bt_panels,
                                int64_t N, float* c_out, void* stream);

/* tri_mul_epilogue: out[i][j] = m_ij * sigmoid(W_g LN_in(z_ij)) * W_o LN_out(C_.[i][j])
 * (C float32 in the result layout of tri_mul_contract, z [N][N][c_z] dtype,
 * out [N][N][c_z] out_dtype). */
int tri_mul_epilogue(tri_mul_handle_t h, const float* c_in, const void* z,
                     const uint8_t* mask, int64_t N, void* out, void* stream);

/* ---------------------------------------------------------------- backward
 *
 * Backward of the contraction, for training (Section 3.1: every distributed
 * module has an explicit backward running the same schedule as its forward).
 * With the operands of tri_mul_contract, C_c = A_c * B_c^T for every channel
 * c, and L a loss with gradient dC = dL/dC:
 *
 *     dA_c = dC_c * B_c          dB_c = dC_c^T * A_c
 *
 * The operands are direction-agnostic: for the incoming update, A and B are
 * the incoming panels (tri_mul_project with TRI_MUL_INCOMING), and the
 * caller maps dA back to a by the same transposition.
 *
 * tri_mul_contract_backward_workspace_size: bytes of device workspace for N
 * tokens: one operand in the panel layout (dC) in the bf16 path, which reads
 * the other operands transposed in place; four (dC and the transposes of dC,
 * A and B) in the fp32 path; 256-byte aligned each.
 * *bytes is a HOST pointer. */
int tri_mul_contract_backward_workspace_size(tri_mul_handle_t h, int64_t N, size_t* bytes);

/* tri_mul_contract_backward:
 *   dC        float32, result layout of tri_mul_contract (N x J x 32 x c floats)
 *   a_panels, b_panels   dtype, panel layout (as written by tri_mul_project)
 *   dA        float32, result layout over (i, k): element (ch, i, k) at
 *             ((i * J + k / 32) * c + ch) * 32 + k % 32; overwritten
 *   dB        float32, result layout over (j, k); overwritten
 *   ws        workspace of >= tri_mul_contract_backward_workspace_size bytes,
 *             256-byte aligned; must not alias any other argument
 * In the bf16 path dC is rounded to bf16 for the products (fp32
 * accumulation).  Returns TRI_MUL_ENOMEM if ws_bytes is too small. */
int tri_mul_contract_backward(tri_mul_handle_t h, const float* dC, const void* a_panels, const void* b_panels,
                              int64_t N, float* dA, float* dB, void* ws, size_t ws_bytes, void* stream);

/* Gradients of the whole update (bf16 storage path), for training.  Given
 * dout = dL/dout (same layout and dtype as the forward's out), the call
 * recomputes the forward from z and returns dz = dL/dz and the gradients of
 * all ten weight tensors:
 *   grads   HOST struct of DEVICE pointers, float32, shapes as in
 *           tri_mul_params_t ([out][in] for the linear maps); overwritten
 *           (sums over all pairs)
 *   dz      [N][N][c_z] dtype; overwritten
 *   ws      workspace of >= tri_mul_backward_workspace_size bytes, 256-byte
 *           aligned; must not alias any other argument
 * Pairs with m_ij = 0 receive dz = 0 and contribute nothing.  Returns
 * TRI_MUL_EUNSUPPORTED for the float32 storage path, TRI_MUL_ENOMEM if
 * ws_bytes is too small. */
typedef struct {
    float* ln_in_w;
    float* ln_in_b;
    float* w_a;
    float* w_ga;
    float* w_b;
    float* w_gb;
    float* w_g;
    float* ln_out_w;
    float* ln_out_b;
    float* w_o;
} tri_mul_grads_t;

int tri_mul_backward_workspace_size(tri_mul_handle_t h, int64_t N, size_t* bytes);
int tri_mul_outgoing_backward(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N, const void* dout,
                              void* dz, const tri_mul_grads_t* grads, void* ws, size_t ws_bytes, void* stream);
int tri_mul_incoming_backward(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N, const void* dout,
                              void* dz, const tri_mul_grads_t* grads, void* ws, size_t ws_bytes, void* stream);

/* The same backward from the forward's saved state instead of recomputing
 * it: a_panels, b_panels -- the direction's operands TRANSPOSED, i.e. the
 * panels tri_mul_project writes for this z and mask with the OPPOSITE
 * direction -- and c_result (result layout, the contraction of the
 * direction, as tri_mul_contract_transposed writes it from those panels, or
 * tri_mul_contract from the direction's own) replace the recomputed
 * projections and contraction; the full calls tri_mul_outgoing /
 * tri_mul_incoming (bf16 storage) leave exactly these in their workspace,
 * at byte offsets 0, P and 2 P with P = tri_mul_panel_size rounded up to a
 * multiple of 256.  Results are
 * identical to tri_mul_outgoing_backward / tri_mul_incoming_backward on the
 * same inputs; the saved tensors are only read and must not alias ws.  Same
 * workspace size, alignment and errors (16-byte aligned saved pointers). */
int tri_mul_outgoing_backward_saved(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N,
                                    const void* a_panels, const void* b_panels, const float* c_result,
                                    const void* dout, void* dz, const tri_mul_grads_t* grads, void* ws,
                                    size_t ws_bytes, void* stream);
int tri_mul_incoming_backward_saved(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N,
                                    const void* a_panels, const void* b_panels, const float* c_result,
                                    const void* dout, void* dz, const tri_mul_grads_t* grads, void* ws,
                                    size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TRI_MUL_H */
