// Host-side launchers of the triangle-multiplication kernels.  Each returns
// hipSuccess or the error hipGetLastError() reported right after the launch.
// Shapes are validated by the C-ABI layer before these are called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace trimul {

// Repacked, device-resident layer parameters (owned by the handle).
struct DeviceWeights {
    // fp32 copies used by the VALU kernels (both storage types)
    float* ln_in_w = nullptr;   // [c_z]
    float* ln_in_b = nullptr;   // [c_z]
    float* ln_out_w = nullptr;  // [c]
    float* ln_out_b = nullptr;  // [c]
    float* proj4 = nullptr;     // [c_z][c][4]: (W_a, W_ga, W_b, W_gb)[c][d] at [d][c][*]
    float* wo_t = nullptr;      // [c][c_z]:   W_o[d][c] at [c][d]
    float* wg_t = nullptr;      // [c_z][c_z]: W_g[d][e] at [e][d]
    // bf16 copies used by the MFMA kernels (bf16 storage only)
    uint16_t* proj_bf = nullptr;  // [4*c][c_z]: rows ordered per 32-channel group g:
                                  // W_a[g], W_ga[g], W_b[g], W_gb[g] (32 rows each)
    uint16_t* epi_bf = nullptr;   // [2*c_z][128]: W_o rows then W_g rows
    uint16_t* epit_bf = nullptr;  // [2*128][c_z]: W_o^T rows then W_g^T rows (backward)
    uint16_t* projt_bf = nullptr; // [c_z][4*c]: row d = W_a[:, d], W_ga[:, d], W_b[:, d], W_gb[:, d] (backward)
    // fp16 copies for the bf16-path projection (K1), each matrix scaled by a
    // power of two 2^s_m and the LayerNorm gain and bias by 2^s_x, so that
    // the largest possible |W x| operand lies in [2^14, 2^15]; the gating
    // undoes the scales (K1Scales).
    uint16_t* proj_h = nullptr;   // [4*c][c_z] fp16 bits, rows as proj_bf, W_m * 2^s_m
    float* ln_in_w_h = nullptr;   // [c_z] gamma * 2^s_x
    float* ln_in_b_h = nullptr;   // [c_z] beta * 2^s_x
    struct K1Scales {
        // a = v * sigmoid(g) from accumulators v' = 2^Sv v, g' = 2^Sg g:
        // a = v' / (2^Sv + 2^(Sv - g log2 e)) = v' * rcp(kv + exp2(g' * cg + Sv))
        float kv_a, cg_a, sv_a;   // 2^Sv, -log2(e) 2^-Sg, Sv of a
        float kv_b, cg_b, sv_b;   // the same for b
    } k1s{};
    float eps = 1e-5f;
    int cus = 256;                // compute units of the device (persistent grids)
    uint8_t* kmask_pad = nullptr; // 0/1 staging of a token mask (k-panel, sequence, or a tile's columns and rows), kMaskStageBytes
};

constexpr int64_t kMaxKPanel = 65536;   // longest k-panel of one block call
constexpr int64_t kMaskStageBytes = 2 * kMaxKPanel + 128;   // size of DeviceWeights::kmask_pad

// Copies mask[0, klen) into dst as 0/1 bytes (mask NULL: all ones) and zero-fills dst up to the next
// multiple of 32 (so the contraction can read whole 4-byte words of it).
hipError_t launch_stage_kmask(const uint8_t* mask, int64_t klen, uint8_t* dst, hipStream_t s);
// Stages a tile's token mask for the epilogue: dst[0, ceil(cols/32)*32) = 0/1 of mask[col0 + k] (zero
// past cols), then dst[ceil(cols/32)*32 + r] = 0/1 of mask[row0 + r] for r < ceil(rows/4)*4 (zero past
// rows); mask NULL: all ones.  dst must hold kMaskStageBytes.
hipError_t launch_stage_tile_mask(const uint8_t* mask, int64_t row0, int64_t rows, int64_t col0, int64_t cols,
                                  uint8_t* dst, hipStream_t s);
// Row-major bf16 panel [nch][rows][ld] -> blocked [nch][ceil(rows/256)][ceil(klen/32)][256][32],
// staged k-mask applied, padding zero.
hipError_t launch_panel_block(const void* P, int64_t rows, int64_t ld, int64_t klen, int nch, const uint8_t* kst,
                              void* dst, hipStream_t s);
// bf16 contraction of blocked operands into a row-major fp32 C [batch][M][N].
hipError_t launch_contract_blocked_rowc(const void* A, const void* B, float* C, int64_t M, int64_t N, int64_t K,
                                        int batch, int accumulate, int cus, hipStream_t s);
// bf16 contraction of blocked operands into the pair-blocked fp32 result layout over (M, N) (a device
// tile's packed accumulator), overwritten or accumulated into.
hipError_t launch_contract_blocked_packed(const void* A, const void* B, float* C, int64_t M, int64_t N, int64_t K,
                                          int batch, int accumulate, int cus, hipStream_t s);
// bf16 contraction of blocked operands, either given as its transpose in the
// panel layout (ta: A[c][i][k] = X[c][k][i], X with K rows and M columns; tb
// likewise with N columns), into the pair-blocked fp32 result layout.
// Supported: (ta, tb) = (0, 1), (1, 1) and (1, 0); accumulate adds into C.
hipError_t launch_contract_transposed(int ta, int tb, const void* A, const void* B, float* C, int64_t M, int64_t N,
                                      int64_t K, int batch, int cus, hipStream_t s, int accumulate = 0);

// Host-side check of the contraction kernel's loads (contract.hip): counts of
// tiles, loads and needed elements visited, and of violations.
struct K2CheckCounts {
    int64_t tiles = 0, loads = 0, elems = 0;
    int64_t bad_tiles = 0;   // tiles taken by no or several (work-group, round) pairs
    int64_t bad_desc = 0;    // loads whose descriptor reaches outside the operand
    int64_t bad_elem = 0;    // needed elements read from the wrong address or not at all
};
// a_mode / b_mode: 0 blocked panel, 1 row-major [batch][rows][ld] (channel stride sA / sB), 2 transposed
// (the operand given as X[k][row] in the panel layout of K rows).  a_bytes / b_bytes: allocation sizes.
void k2_check_loads(int a_mode, int b_mode, int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t sA,
                    int64_t sB, int batch, uint64_t a_bytes, uint64_t b_bytes, int grid, int all_channels,
                    K2CheckCounts& n);
// The same for the accesses to a pair-blocked C of M rows, N columns and `batch` channels (the result layout,
// c_bytes allocated): every load / store descriptor inside the allocation, every accessed element at the
// layout's address, every element (row < M, column < N) accessed exactly once (loads counts the 64-lane
// register groups visited).
void k2_check_c(int64_t M, int64_t N, int batch, uint64_t c_bytes, int all_channels, K2CheckCounts& n);

struct EpilogueArgs {
    const float* C;      // fp32 contraction result: pair-blocked (cblocked) or [c][rows][ldc]
    int cblocked;        // C in the pair-blocked result layout (common.h)
    int64_t ldc;         // row stride of C (elements), row-major C only
    int64_t sc;          // channel stride of C (elements), row-major C only
    const void* z;       // [rows][cols][c_z] pair tensor (same tile as C)
    const uint8_t* mask; // token mask over global indices, or null
    int64_t row0, col0;  // global token index of tile row 0 / column 0
    int64_t rows, cols;
    void* out;           // [rows][cols][c_z]
};

// K1: LN_in + gated projections + pair mask -> channel-major operands A, B in
// the blocked panel layout (common.h) of N rows and K = N.  Padding rows are
// left untouched; the k padding of a row's last k-step is written with zeros.
// The bf16 projection of an M x K operand pair (A, B in the blocked layout of
// panel_geom(M, K)): operand row i, contraction index k is pair (i, k) of z
// (outgoing) or (k, i) (incoming), z rows ldz pairs apart; tmask holds the
// staged 0/1 bytes of the k-range at [0, ceil(K/32)*32) and of operand row i
// at rmoff + i.
hipError_t launch_project_mfma(const DeviceWeights& w, const void* z, int64_t ldz, const uint8_t* tmask, int64_t rmoff,
                               int64_t M, int64_t K, int incoming, void* A, void* B, hipStream_t s);
hipError_t launch_project(int dtype, const DeviceWeights& w, const void* z, const uint8_t* mask,
                          int64_t N, int incoming, void* A, void* B, hipStream_t s);

// K2: C[b] (+)= A[b] * diag(kmask) * B[b]^T for b < batch.
// blocked != 0: A, B in the blocked panel layout of M (N) rows and K columns
// (lda, ldb, sA, sB unused) and C in the pair-blocked result layout (ldc, sC
// unused); blocked == 0: A [b][M][lda], B [b][N][ldb], C [b][M][ldc] (stride sC).
hipError_t launch_contract(int dtype, int blocked, const void* A, const void* B, float* C, int64_t M,
                           int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc, int64_t sA,
                           int64_t sB, int64_t sC, int batch, int accumulate, const uint8_t* kmask, int cus,
                           hipStream_t s);

// K3: LN_out + output projection + sigmoid gate + pair mask -> out [rows][cols][c_z].
hipError_t launch_epilogue(int dtype, int out_dtype, const DeviceWeights& w, const EpilogueArgs& a,
                           hipStream_t s);

// Backward of the contraction: the fp32 result layout -> a panel (dtype
// elements), and the per-channel panel transpose X_c[i][k] -> X_c[k][i].
hipError_t launch_result_to_panel(int dtype, const float* R, void* P, int64_t N, int cus, hipStream_t s);
hipError_t launch_panel_transpose(int dtype, const void* X, void* Y, int64_t N, int cus, hipStream_t s);

// Layer backward (bf16 storage).  Unit blocks: per unit of 32 pairs a bf16
// [128][32] block of one per-pair quantity (see backward.hip).
struct BackwardBlocks {
    bf16_t *du, *y, *dgg, *xe;         // from the epilogue backward
    bf16_t *dpa, *dga, *dpb, *dgb, *xp; // from the projection backward
};
// Persistent grid: min(units, per_cu * compute units).
int backward_grid(int64_t units, int cus, int per_cu);
hipError_t launch_epilogue_backward(int out_dtype, const DeviceWeights& w, const float* C, const void* z,
                                    const uint8_t* mask, const void* dout, int64_t N, void* dCp, float* dxg,
                                    const BackwardBlocks& bb, float* partial, int grid, hipStream_t s);
hipError_t launch_projection_backward(const DeviceWeights& w, const void* z, const uint8_t* mask, int64_t N,
                                      int incoming, const float* dA, const float* dB, const float* dxg, void* dz,
                                      const BackwardBlocks& bb, float* partial, int grid, hipStream_t s);
hipError_t launch_wgrad(const bf16_t* U, const bf16_t* V, int64_t N, float* partial, int grid, hipStream_t s);
// Four weight gradients sharing V: partial[o][grid][128][128] for U[o] V^T, o = 0..3.
hipError_t launch_wgrad4(const bf16_t* const U[4], const bf16_t* V, int64_t N, float* partial, int grid,
                         hipStream_t s);
hipError_t launch_sum_parts(const float* in, int parts, int64_t stride, int n, float* out, hipStream_t s);

// Outer product mean (opm.hip).  Pack: tokens [tok0, tok0 + ntok) and
// sequences [s0, s0 + slen) of a [S][n_total][32] bf16 tensor, masked, into
// the transposed operand of the sums -- the blocked panel of slen rows and
// ntok * 32 columns, X[s][token * 32 + c] -- and the 0/1 mask into the
// (plain) blocked panel of ntok rows and K = slen.  Epilogue: out[rows][cols][128]
// from the sums O (result layout, [rows * 32][cols * 32]) and the counts
// (result layout, [rows][32 * ceil(cols / 32)]).
hipError_t launch_opm_pack(const void* a, const uint8_t* mask, int64_t n_total, int64_t tok0, int64_t ntok,
                           int64_t s0, int64_t slen, void* P, void* Mp, hipStream_t s);
hipError_t launch_opm_epilogue(int out_dtype, const float* O, const float* cnt, int64_t rows, int64_t cols,
                               const uint16_t* wo, const float* bo, void* out, int cus, hipStream_t s);

// Triangle attention core (triattn.hip): rows x heads x ceil(N / 128)
// work-groups over keys [k0, kend); q, k, v [rows][N][H][32] bf16, bias
// [H][N][ldb] bf16 (ldb % 8 == 0, k0 % 8 == 0), mask [N] or null.  State
// (A [rows][N][H][32], M and L [rows][H][N], fp32) is read when load_state and
// written unless finish; finish writes out [rows][N][H][32] (fp32 or bf16).
hipError_t launch_triattn(int out_dtype, const void* q, const void* k, const void* v, const void* bias,
                          const uint8_t* mask, int64_t rows, int64_t N, int H, int64_t ldb, int64_t k0, int64_t kend,
                          float* stA, float* stM, float* stL, int load_state, int finish, void* out, hipStream_t s);

}  // namespace trimul
