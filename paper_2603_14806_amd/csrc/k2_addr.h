// Loader addressing of the bf16 contraction kernel (k2_contract_ws): the
// tile order, and for every direct-to-LDS load the buffer descriptor (base
// and range) and the byte offset within it.  The kernel computes its loads
// with these functions, and so does the host-side checker
// (k2_check_loads in contract.hip), which walks every load of a launch and
// verifies that each descriptor lies inside its operand's allocation and that
// every element a tile needs arrives from the address the operand's layout
// gives it.
//
// Every offset travels in the lane offset (voffset); the scalar offset of the
// loads is always 0.  A load whose part of the tile lies outside the operand
// (rows past the panel, a transposed operand's column blocks past its last
// one) gets a range that excludes it, or the empty descriptor, so it reads
// zeros without touching memory.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace trimul {

constexpr int kK2Tile = 256;   // output tile side (rows of A and of B per tile)
constexpr int kK2BK = 32;      // k per step
constexpr int kK2Row = kK2BK * 2;          // bytes of one operand row of a step in LDS
constexpr int kK2Loaders = 4;              // loader waves
constexpr int kK2LoadsPerOperand = 4;      // loads per loader wave, operand and step
// The blocked layout holds one 256-row x 32-k block per panel block: a tile's
// k-step is one block only when the tile side and the step equal the block's.
static_assert(kK2Tile == kBlkRows && kK2BK == kBlkK, "a K2 tile step must be exactly one panel block");
static_assert(kK2Loaders * kK2LoadsPerOperand * 16 == kK2Tile, "loader waves cover the tile's rows");

// Operand layouts.
enum { kK2Blocked = 0, kK2RowMajor = 1, kK2Transposed = 2 };

struct K2Operand {
    int mode;        // kK2Blocked, kK2RowMajor or kK2Transposed
    int rows;        // logical rows (M for A, N for B)
    int K;           // contraction length
    int ld;          // kK2RowMajor: elements between rows
    int64_t stride;  // kK2RowMajor: elements between channels
};

struct K2Desc {
    int64_t base;    // element offset of the descriptor's base from the operand start
    uint32_t range;  // bytes covered (0: the empty descriptor)
};

// ------------------------------------------------------------- tile order
//
// Persistent grid of G work-groups.  Work-group wg runs on XCD wg % 8 (the
// dispatcher deals work-groups round-robin over the 8 XCDs); perm renumbers
// them so that the 32 work-groups of one XCD hold consecutive numbers.  In
// round it, work-group perm takes logical tile it * G + perm.  Logical tiles
// run channel by channel; within a channel in groups of 4 tile rows, and
// within a group column-major, so 32 consecutive tiles form a 4 x 8 block
// whose A row panels and B column panels the XCD's L2 shares.
__host__ __device__ __forceinline__ int k2_perm(int wg, int G) {
    return (G & 7) == 0 ? (wg & 7) * (G >> 3) + (wg >> 3) : wg;
}
__host__ __device__ __forceinline__ int k2_my_tiles(int perm, int G, int total) {
    return perm < total ? (total - 1 - perm) / G + 1 : 0;
}
struct K2Tile {
    int ch, m0, n0;
};
__host__ __device__ __forceinline__ K2Tile k2_decode(int L, int tiles_m, int tiles_n) {
    constexpr int GR = 4;
    const int tiles = tiles_m * tiles_n;
    K2Tile t;
    t.ch = L / tiles;
    const int rem = L - t.ch * tiles;
    const int gid = rem / (GR * tiles_n);
    const int first_m = gid * GR;
    const int gsz = tiles_m - first_m < GR ? tiles_m - first_m : GR;
    const int in_g = rem - gid * GR * tiles_n;
    t.m0 = (first_m + in_g % gsz) * kK2Tile;
    t.n0 = (in_g / gsz) * kK2Tile;
    return t;
}

// ------------------------------------------------------------- loads
//
// Loader wave lw (0..3) issues, per operand and step, loads jj = 0..3, each
// 64 lanes x 16 bytes into LDS rows 64 lw + 16 jj .. + 15 of the operand's
// half of the stage (lane i writes bytes 16 i .. + 15 of that 1 KB piece).
//
// Blocked / row-major: LDS row r holds operand row t0 + r of the step, its
// 16-byte chunk q (k = 32 kt + 8 q .. + 7) at slot q ^ ((r >> 2) & 3); lane i
// fills row r = 64 lw + 16 jj + i / 4, slot i % 4.
// Transposed (the operand is given as X with X[k][row] = operand[row][k]):
// the 1 KB piece (2 lw + jj / 2, jj % 2) is rows 16 (jj % 2) .. + 15 of
// the step (k = 32 kt + those) of the tile's 32-column block 2 lw + jj / 2, 64
// bytes per k row, no swizzle.

// Byte offset of lane `lane` of loader wave lw within the step's first piece
// (the part of the lane offset that does not change from load to load).
__host__ __device__ __forceinline__ uint32_t k2_lane_off(const K2Operand& op, int lw, int lane) {
    if (op.mode == kK2Transposed) return (uint32_t)(lane * 16);
    const int row = lw * 64 + (lane >> 2);
    const int chunk = (lane & 3) ^ ((lane >> 4) & 3);   // the k chunk that lands in slot lane % 4
    const int rs = op.mode == kK2Blocked ? kK2BK : op.ld;
    return (uint32_t)((row * rs + chunk * 8) * 2);
}

// Number of 256-row tiles of the X panel (transposed operand: X has K rows)
// and its 32-column blocks.
__host__ __device__ __forceinline__ int k2_tr_blocks(const K2Operand& op) { return (op.rows + 31) / 32; }

// Descriptor of the operand part that tile rows t0 .. t0 + 255 read in step
// kt: for the blocked and row-major layouts the same for every step of a
// tile, for a transposed operand the 256-row tile of X that holds the step.
__host__ __device__ __forceinline__ K2Desc k2_desc(const K2Operand& op, int ch, int t0, int kt) {
    const int nk = (op.K + kK2BK - 1) / kK2BK;
    const int tiles = (op.rows + kK2Tile - 1) / kK2Tile;
    K2Desc d;
    if (op.mode == kK2Blocked) {
        d.base = ((int64_t)ch * tiles + t0 / kK2Tile) * nk * (kK2Tile * kK2BK);
        d.range = (uint32_t)nk * (uint32_t)(kK2Tile * kK2BK * 2);
    } else if (op.mode == kK2RowMajor) {   // rows past the operand fall outside the range
        d.base = (int64_t)ch * op.stride + (int64_t)t0 * op.ld;
        const int live = op.rows - t0 < kK2Tile ? op.rows - t0 : kK2Tile;
        d.range = (uint32_t)live * (uint32_t)op.ld * 2u;
    } else {
        const int xs = k2_tr_blocks(op), xt = (op.K + kK2Tile - 1) / kK2Tile;
        d.base = ((int64_t)ch * xt + (kt >> 3)) * xs * (kK2Tile * kK2BK);
        d.range = (uint32_t)xs * (uint32_t)(kK2Tile * kK2BK * 2);
    }
    return d;
}

// Wave-uniform byte offset of load jj of loader wave lw in step kt (added to
// k2_lane_off).  Returns false when the whole load lies outside the operand
// (a transposed operand's column block past its last one): the load then
// goes to the empty descriptor.
__host__ __device__ __forceinline__ bool k2_load_off(const K2Operand& op, int t0, int kt, int lw, int jj,
                                                      uint32_t& off) {
    if (op.mode == kK2Transposed) {
        const int cb = (t0 >> 5) + 2 * lw + (jj >> 1);
        off = (uint32_t)cb * (uint32_t)(kK2Tile * kK2BK * 2) + (uint32_t)((kt & 7) * 32 + 16 * (jj & 1)) * kK2Row;
        return cb < k2_tr_blocks(op);
    }
    if (op.mode == kK2Blocked) {
        off = (uint32_t)(jj * 16 * kK2BK * 2) + (uint32_t)kt * (uint32_t)(kK2Tile * kK2BK * 2);
    } else {
        off = (uint32_t)jj * (uint32_t)(16 * op.ld * 2) + (uint32_t)kt * kK2Row;
    }
    return true;
}

// LDS byte offset (within the operand's half of a stage) of load jj of
// loader wave lw: the same for every layout.
__host__ __device__ __forceinline__ uint32_t k2_lds_off(int lw, int jj) {
    return (uint32_t)(lw * 64 + 16 * jj) * kK2Row;
}

// ------------------------------------------------------------- pair-blocked C
//
// The result C of nch channels in the pair-blocked layout (result_off):
// element (ch, i, j) at ((i * J + j / 32) * nch + ch) * 32 + j % 32 floats,
// J = ceil(N / 32); a row is crs = J * nch * 32 floats long.  MFMA wave w
// (0..7) of a tile owns its rows 64 (w / 2) .. + 63 and columns
// 128 (w % 2) .. + 127, as eight 32 x 32 blocks x = 4 (rows / 32) + column
// block; in the accumulator layout lane l holds column l % 32 and, in
// register r, row 8 (r / 4) + 4 (l / 32) + r % 4 of a block.  Each of the
// wave's four column blocks goes through one descriptor from the block's
// first element whose range covers the rows < M, so that rows past M fall
// outside it; a column block past C's last gets the empty descriptor (its
// memory belongs to the next row).  Columns past N inside C's last block
// are the layout's padding and are accessed like the rest.  The byte offset
// is the lane part (k2_c_lane_off) plus the wave-uniform part of block x,
// register r (k2_c_reg_off); both travel in the lane offset.
__host__ __device__ __forceinline__ uint32_t k2_c_row_floats(int N, int nch) {
    return (uint32_t)((N + kResJ - 1) / kResJ) * (uint32_t)nch * kResJ;
}
__host__ __device__ __forceinline__ K2Desc k2_c_desc(int M, int N, int nch, const K2Tile& t, int wave, int j) {
    const int jblocks = (N + kResJ - 1) / kResJ;
    const int wrow0 = t.m0 + (wave >> 1) * 64, wcol0 = t.n0 + (wave & 1) * 128;
    const int nrows = M - wrow0 < 64 ? M - wrow0 : 64;
    const bool live = nrows > 0 && wcol0 / kResJ + j < jblocks;
    K2Desc d;
    d.base = live ? result_off(jblocks, nch, t.ch, wrow0, wcol0 + kResJ * j) : 0;
    d.range = live ? ((uint32_t)(nrows - 1) * k2_c_row_floats(N, nch) + kResJ) * 4u : 0u;
    return d;
}
__host__ __device__ __forceinline__ uint32_t k2_c_lane_off(uint32_t crs, int lane) {
    return (4u * (uint32_t)(lane >> 5) * crs + (uint32_t)(lane & 31)) * 4u;
}
__host__ __device__ __forceinline__ uint32_t k2_c_reg_off(uint32_t crs, int x, int r) {
    return (uint32_t)((x >> 2) * 32 + 8 * (r >> 2) + (r & 3)) * crs * 4u;
}
// The logical row and column of that element (for the host check).
__host__ __device__ __forceinline__ void k2_c_elem(const K2Tile& t, int wave, int lane, int x, int r, int& row, int& col) {
    row = t.m0 + (wave >> 1) * 64 + (x >> 2) * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
    col = t.n0 + (wave & 1) * 128 + (x & 3) * 32 + (lane & 31);
}

}  // namespace trimul
