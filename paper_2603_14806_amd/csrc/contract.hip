// K2: the per-channel contraction of Eq. 2 / Eq. 3 (Section 3.3), which the
// paper describes as a batched matrix multiplication.  After K1's layout
// change both directions are the same "NT" product per hidden channel c:
//
//     C[c][i][j] (+)= sum_k A[c][i][k] * m_k * B[c][j][k]
//
// m_k is an optional token mask over k (used by the block path, where the
// panels arrive unmasked).  The bf16 path runs on gfx950 matrix cores
// (v_mfma_f32_32x32x16_bf16, fp32 accumulation); the fp32 path is a plain
// LDS-tiled VALU kernel.
#include <vector>

#include "common.h"
#include "k2_addr.h"
#include "kernels.h"

namespace trimul {
namespace {

// ---------------------------------------------------------------- bf16 MFMA
//
// Persistent kernel, one work-group per CU, looping over 256 x 256 output
// tiles.  The k loop runs in steps of 32 through an LDS ring of 32 KB stages
// filled by direct-to-LDS buffer loads (no VGPR staging) several steps ahead
// of the step being multiplied; the ring flows straight from one output
// tile into the next.
//
// Tile order: in round r the work-groups on XCD x take 32 consecutive
// logical tiles, i.e. a 4 x 8 block of one channel, so the A row panels and B
// column panels of a block are fetched once into that XCD's L2 and served to
// the 32 CUs that share it.
//
// LDS layout of a stage: 256 A rows then 256 B rows of 32 bf16 (64 bytes =
// 4 chunks of 16 bytes); chunk q of row r sits at slot q ^ ((r >> 2) & 3).
// gfx950's LDS has 64 banks and serves a 16-byte-per-lane read 16 lanes per
// cycle; the 16 rows those lanes read then cover all 64 banks.
constexpr int BN = 256, BK = 32;
constexpr int ROWB = BK * 2;                    // 64 bytes per row per stage
constexpr int B_ST = BN * ROWB;                 // 16 KB
constexpr int kLdsBytes = 160 * 1024;           // gfx950 LDS per work-group

// Eight bf16 of an MFMA operand from a row-major [k][32] LDS block through
// two ds_read_b64_tr_b16 (k values 0-3, then 4-7 from four rows further on).
typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef short v8i16_t __attribute__((ext_vector_type(8)));
__device__ __forceinline__ bf16x8_t lds_read_tr8(const char* p) {
    typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;
    const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(p));
    const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(p + 4 * ROWB));
    const v8i16_t v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8_t, v);
}

// ------------------------------------------- bf16 MFMA, 8 + 4 specialised waves
//
// The contraction with the loads taken off the MFMA waves: 12 waves per
// work-group (three per SIMD); waves 0-7 each own a 64 x 128 sub-tile (2 x 4
// MFMA blocks, 128 accumulator registers) and issue only LDS reads and
// MFMAs, waves 8-11 issue all 32 direct-to-LDS loads of a k-step (64 A rows
// and 64 B rows each) and wait for them, so a load that stalls in a busy L2
// never stops a matrix-core stream.  The one barrier per k-step hands
// filled stages from the loaders to the MFMA waves and a consumed one back;
// at barrier s steps s and s + 1 are complete, and the MFMA waves read step
// s + 1's first operands behind step s's last MFMAs.
//
// Operands either blocked (one tile's k-step is a contiguous 16 KB block:
// the full update, the outer product mean, and a device tile's panels
// repacked by k_panel_block) or row-major (a device tile's caller panels
// [ch][rows][ld]); C either in the pair-blocked result layout (the full
// update) or row-major [ch][rows][ldc] (a device tile's accumulator).  k values that must not reach the sums -- masked by the
// optional k-mask, or past K in the last step (row-major padding columns
// hold arbitrary data) -- are zeroed in LDS by the loader waves, in the rows
// each loaded, before the barrier that publishes the stage: only steps that
// hold such k pay, and the MFMA waves never mask.
// LDS ring of 5 stages, swizzle and tile order as described above.
//
// Transposed operands (TA / TB, blocked only, no k-mask): the operand is
// given as its transpose X in the panel layout, A[c][i][k] = X[c][k][i], so
// the products of the backward, dC B and dC^T A, run without transposing
// panels in memory.  A k-step of a 256-wide tile is then the 32 rows k of
// eight 32-column blocks of X: eight contiguous 2 KB pieces, copied to LDS
// as they are (block b of the tile at 2 KB b, 64 bytes per row k, no
// swizzle).  The MFMA waves read such an operand with ds_read_b64_tr_b16:
// lanes 16 g + 4 i + a (g < 4, i < 4, a < 4) address row 8 (g >> 1) + i,
// columns 16 (g & 1) + 4 a .. + 3 of a block, and lane 16 g + 4 a + b receives
// element b of the four chunks lanes 16 g + a, + 4, + 8, + 12 address, i.e.
// column 16 (g & 1) + 4 a + b of rows 8 (g >> 1) .. + 3 -- the MFMA operand
// layout, 4 of its 8 k values; a second read 4 rows further gives the rest.
// A half-wave reads 256 contiguous bytes: no bank conflicts.
// Round pacing.  The work-groups of one XCD share their round's A row
// panels and B column panels through that XCD's L2 only while they stream
// the same k range; left alone they drift apart (measured: up to ~100 us,
// about 100 k-steps, within a few rounds, far beyond the ~20 k-steps of
// operand traffic the L2 holds), and every lagging tile then refetches its
// panels from memory.  So at the start of every full round each work-group
// counts in on its XCD's counter and waits until all G / 8 of them have (a
// bounded wait: 20 us, after which it goes on anyway -- pacing changes only
// where the data comes from, never the results).  One 128-byte line per XCD;
// reset by k_pace_reset before every paced launch.  Concurrent contraction
// launches on one device share the counters and then mostly wait the bound.
constexpr int kPaceLine = 32;   // counters per 128-byte line
__device__ unsigned int g_k2_pace[8 * kPaceLine];
__global__ void k_pace_reset() {
    if (threadIdx.x < 8 * kPaceLine) g_k2_pace[threadIdx.x] = 0u;
}

template <bool BLOCKED, bool KMASK, bool CBLOCKED, bool TA = false, bool TB = false>
__global__ __attribute__((amdgpu_flat_work_group_size(768, 768), amdgpu_waves_per_eu(3, 3)))
void k2_contract_ws(const bf16_t* __restrict__ A, const bf16_t* __restrict__ B, float* __restrict__ C, int M,
                    int N, int K, int lda, int ldb, int64_t ldc, int64_t sA, int64_t sB, int64_t sC, int tiles_m,
                    int tiles_n, int total, int accumulate, const uint8_t* __restrict__ kmask, int pace) {
    constexpr int BM = kK2Tile, MI = 2;
    constexpr int A_ST = BM * ROWB, ST_BYTES = A_ST + B_ST;
    constexpr int STAGES = kLdsBytes / ST_BYTES;  // 5
    constexpr int LOADS = 2 * kK2LoadsPerOperand;  // direct-to-LDS loads per loader wave per step
    static_assert(!(TA || TB) || (BLOCKED && !KMASK), "transposed operands are blocked and unmasked");
    // a blocked operand's k-step must be exactly one panel block (256 rows x 32 k)
    static_assert(!BLOCKED || (BM == kBlkRows && BN == kBlkRows && BK == kBlkK), "blocked tiles are panel blocks");
    static_assert(BN == kK2Tile && BK == kK2BK && ROWB == kK2Row, "loader addressing assumes this tile");
    __shared__ __attribute__((aligned(16))) char smem[STAGES * ST_BYTES];

    const int G = gridDim.x, wg = blockIdx.x;
    const int perm = k2_perm(wg, G);
    const int my_tiles = k2_my_tiles(perm, G, total);
    const int nk = (K + BK - 1) / BK;
    const int steps = my_tiles * nk;
    const int tiles = tiles_m * tiles_n;
    const int nchan = total / tiles;

    const int t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);   // 0 .. 11
    const uint32_t lds_base = lds_addr(smem);

    if (wave >= 8) {
        // Loader wave lw: rows 64 lw .. 64 lw + 63 of the A and B halves of a
        // stage as four 16-row loads each (k2_addr.h).  Every offset is in the
        // lane offset; the scalar offset is 0.
        const int lw = wave - 8;
        const K2Operand opa{TA ? kK2Transposed : BLOCKED ? kK2Blocked : kK2RowMajor, M, K, lda, sA};
        const K2Operand opb{TB ? kK2Transposed : BLOCKED ? kK2Blocked : kK2RowMajor, N, K, ldb, sB};
        const uint32_t la = k2_lane_off(opa, lw, lane), lb = k2_lane_off(opb, lw, lane);
        int l_it = 0, l_kt = 0, l_stage = 0, l_ch = 0, l_m0 = 0, l_n0 = 0;
        const v4i_t rnone = buffer_desc(A, 0u);
        v4i_t ra = rnone, rb = rnone;
        auto desc = [&](const bf16_t* X, const K2Operand& op, int t0, int kt) {
            const K2Desc d = k2_desc(op, l_ch, t0, kt);
            return buffer_desc(X + d.base, d.range);
        };
        auto load_tile = [&]() {
            if (pace && lw == 0 && l_it > 0 && (l_it + 1) * G <= total) {   // every full round but the first
                unsigned int* cnt = &g_k2_pace[(wg & 7) * kPaceLine];
                const unsigned int target = (unsigned int)l_it * (unsigned int)(G >> 3);
                if (lane == 0) atomicAdd(cnt, 1u);
                const uint64_t t0 = __builtin_amdgcn_s_memrealtime();   // 100 MHz
                while (true) {
                    const unsigned int v = __builtin_amdgcn_readfirstlane(
                        __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
                    if (v >= target || __builtin_amdgcn_s_memrealtime() - t0 > 2000u) break;
                    __builtin_amdgcn_s_sleep(1);
                }
            }
            const K2Tile tl = k2_decode(l_it * G + perm, tiles_m, tiles_n);
            l_ch = tl.ch;
            l_m0 = tl.m0;
            l_n0 = tl.n0;
            if (!TA) ra = desc(A, opa, l_m0, 0);
            if (!TB) rb = desc(B, opb, l_n0, 0);
        };
        auto issue_step = [&](bool live) {
            const uint32_t st = lds_base + (uint32_t)(l_stage * ST_BYTES);
            const v4i_t rta = TA ? desc(A, opa, l_m0, l_kt) : ra, rtb = TB ? desc(B, opb, l_n0, l_kt) : rb;
#pragma unroll
            for (int j = 0; j < LOADS; ++j) {   // j < 4: A loads, j >= 4: B loads
                const bool isb = j >= kK2LoadsPerOperand;
                const int jj = j % kK2LoadsPerOperand;
                uint32_t off;
                const bool in = k2_load_off(isb ? opb : opa, isb ? l_n0 : l_m0, l_kt, lw, jj, off);
                const uint32_t dst = st + (isb ? A_ST : 0) + k2_lds_off(lw, jj);
                lds_load16((live && in) ? (isb ? rtb : rta) : rnone, (isb ? lb : la) + off, 0u, dst);
            }
        };
        auto advance = [&]() {
            l_stage = l_stage == STAGES - 1 ? 0 : l_stage + 1;
            if (++l_kt == nk) {
                l_kt = 0;
                if (++l_it < my_tiles) load_tile();
            }
        };
        // Dead-k bitmaps of the k-mask (bit k of step kt set if k-mask byte
        // kt * 32 + k is 0), computed once before any load is in flight:
        // lane l holds steps l + 64 j in mwords[j] (K <= 65536 -> j < 32).
        uint32_t mwords[KMASK ? 32 : 1];
        if (KMASK) {
            const uint32_t* km4 = reinterpret_cast<const uint32_t*>(kmask);   // staged: 0/1 bytes, padded to 32
#pragma unroll
            for (int j = 0; j < 32; ++j) {
                const int kt = lane + 64 * j;
                uint32_t wbits = 0;
                if (kt < nk) {
#pragma unroll
                    for (int d = 0; d < 8; ++d) {
                        const uint32_t m4 = km4[kt * 8 + d];
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (((m4 >> (8 * e)) & 0xffu) == 0) wbits |= 1u << (4 * d + e);
                    }
                }
                mwords[j] = wbits;
            }
        }
        // Zero, in this wave's 64 A and 64 B rows of step u's stage, the k
        // values of the step that are masked out or past K.
        auto zero_dead = [&](int u) {
            const int kt = u % nk;
            const int kv = K - kt * BK;                   // valid k of the step
            uint32_t bits = kv >= BK ? 0u : ~((1u << kv) - 1u);
            if (KMASK) {
                uint32_t wsel = 0;
#pragma unroll
                for (int j = 0; j < 32; ++j) wsel = (j == (kt >> 6)) ? mwords[j] : wsel;
                bits |= (uint32_t)__builtin_amdgcn_readlane((int)wsel, kt & 63);
            }
            bits = __builtin_amdgcn_readfirstlane(bits);
            if (bits == 0) return;
            char* st = smem + (u % STAGES) * ST_BYTES;
            const int r = lw * 64 + lane;                 // this lane's row of the A and of the B block
            if (TA || TB) {   // in a transposed operand the row is k = lane % 32 of a column block
                if ((bits >> (lane & 31)) & 1u) {
                    const uint4 zero = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        if (TA) *reinterpret_cast<uint4*>(st + r * ROWB + 16 * q) = zero;
                        if (TB) *reinterpret_cast<uint4*>(st + A_ST + r * ROWB + 16 * q) = zero;
                    }
                }
                if (TA && TB) return;
            }
            const int sw = (r >> 2) & 3;
            while (bits) {
                const int k = __builtin_ctz(bits);
                bits &= bits - 1;
                const uint32_t o = (uint32_t)(r * ROWB + ((((k >> 3) ^ sw)) << 4) + (k & 7) * 2);
                if (!TA) *reinterpret_cast<bf16_t*>(st + o) = 0;
                if (!TB) *reinterpret_cast<bf16_t*>(st + A_ST + o) = 0;
            }
        };
        if (my_tiles > 0) load_tile();
        const int pro = min(STAGES - 1, steps);
        for (int s0 = 0; s0 < pro; ++s0) {
            issue_step(true);
            advance();
        }
        for (int s = 0; s < steps; ++s) {
            // steps s and s + 1 complete at barrier s; later ones in flight.
            // (Waits with a memory clobber: the LDS zeroing below must not
            // be moved above them.)
            const int ahead = min(STAGES - 3, steps - 2 - s);
            if (ahead >= 2) wait_vmcnt_pinned<2 * LOADS>();
            else if (ahead == 1) wait_vmcnt_pinned<LOADS>();
            else wait_vmcnt_pinned<0>();
            if (s == 0) zero_dead(0);
            if (s + 1 < steps) zero_dead(s + 1);
            __syncthreads();
            const bool fetch = s + STAGES - 1 < steps;
            issue_step(fetch);
            if (fetch) advance();
        }
        wait_vmcnt_pinned<0>();
        return;
    }

    const int wm = wave >> 1, wn = wave & 1;                   // rows 64 wm, columns 128 wn
    // The matrix-core waves issue ahead of the loader wave that shares their
    // SIMD (instruction-issue priority inside the work-group; 1% faster than
    // equal priority, the reverse 0.5% slower).
    __builtin_amdgcn_s_setprio(1);
    const int rl = lane & 31, hi = lane >> 5;
    const int q = (rl >> 2) & 3;
    uint32_t rdA[2], rdB[2];
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
        const uint32_t x = (uint32_t)(((2 * sub + hi) ^ q) << 4);
        rdA[sub] = (wm * 64 + rl) * ROWB + x;
        rdB[sub] = A_ST + (wn * 128 + rl) * ROWB + x;
    }
    // transposed operands: this lane's address in a column block
    const int tg = lane >> 4;
    const uint32_t trb = (uint32_t)((8 * (tg >> 1) + ((lane >> 2) & 3)) * ROWB + (16 * (tg & 1) + 4 * (lane & 3)) * 2);
    // operand i (A) / j (B) of sub-step sub from the stage at st
    auto opA = [&](const char* st, int sub, int i) -> bf16x8_t {
        if constexpr (TA) return lds_read_tr8(st + trb + (2 * wm + i) * 2048 + sub * 16 * ROWB);
        else return *reinterpret_cast<const bf16x8_t*>(st + rdA[sub] + i * 32 * ROWB);
    };
    auto opB = [&](const char* st, int sub, int j) -> bf16x8_t {
        if constexpr (TB) return lds_read_tr8(st + A_ST + trb + (4 * wn + j) * 2048 + sub * 16 * ROWB);
        else return *reinterpret_cast<const bf16x8_t*>(st + rdB[sub] + j * 32 * ROWB);
    };
    // Pair-blocked C (CBLOCKED): descriptors and offsets from k2_addr.h
    // (rows past M fall outside a block's descriptor: loads read 0, stores
    // are dropped).
    const uint32_t crs = k2_c_row_floats(N, nchan);
    const uint32_t cvo = k2_c_lane_off(crs, lane);
    auto cdesc = [&](const K2Tile& tl, __amdgpu_buffer_rsrc_t* rc) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const K2Desc d = k2_c_desc(M, N, nchan, tl, wave, j);
            rc[j] = make_rsrc(C + d.base, d.range);
        }
    };
    // byte offset of register r of 32 x 32 block x from the lane's base vo.
    // Each use site passes a fresh copy of the base (opaque to the
    // compiler), so that the 32 row offsets are formed where they are used
    // instead of being hoisted out of the tile loop and kept in registers
    // the accumulators need.
    auto coff = [&](uint32_t vo, int x, int r) -> uint32_t { return vo + k2_c_reg_off(crs, x, r); };
    auto fresh = [](uint32_t v) {
        asm volatile("" : "+v"(v));
        return v;
    };
    int c_stage = 0;
    for (int it = 0; it < my_tiles; ++it) {
        bf16x8_t a0[MI], b0[4];  // sub-step 0 operands, read one step ahead within a tile
        f32x16_t acc[MI][4];
        if (CBLOCKED && accumulate) {
            // accumulating: the accumulators start from C, all 128 loads
            // issued together and waited for once (one HBM round trip per
            // tile instead of one per 32 x 32 block at the end)
            __amdgpu_buffer_rsrc_t rc[4];
            cdesc(k2_decode(it * G + perm, tiles_m, tiles_n), rc);
            const uint32_t vo = fresh(cvo);
#pragma unroll
            for (int x = 0; x < 4 * MI; ++x)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    acc[x >> 2][x & 3][r] =
                        __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rc[x & 3], coff(vo, x, r), 0, 0));
            wait_vmcnt_pinned<0>();
        } else {
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
        }

        // a tile's first step: barrier, then its sub-step 0 operands (nothing
        // is read ahead across the C stores)
        __syncthreads();
#pragma unroll
        for (int j = 0; j < 4; ++j)
            b0[j] = opB(smem + c_stage * ST_BYTES, 0, j);
#pragma unroll
        for (int i = 0; i < MI; ++i)
            a0[i] = opA(smem + c_stage * ST_BYTES, 0, i);
        for (int kt = 0; kt < nk; ++kt) {
            if (kt > 0) __syncthreads();
            const char* st = smem + c_stage * ST_BYTES;
            c_stage = c_stage == STAGES - 1 ? 0 : c_stage + 1;
            const char* stn = smem + c_stage * ST_BYTES;             // the next step
            bf16x8_t a1[MI], b1[4];
#pragma unroll
            for (int x = 0; x < 4 * MI; ++x) {
                const int i = x >> 2, j = x & 3;
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[i], b0[j], acc[i][j], 0, 0, 0);
                const int y = x - 2;   // reads of sub-step 1 start after the first two MFMAs
                if (y >= 0 && y < 4) b1[y] = opB(st, 1, y);
                else if (y >= 4 && y < 4 + MI) a1[y - 4] = opA(st, 1, y - 4);
            }
            // sub-step 1; after MFMA x, the operand read x - 2 of the next
            // step's sub-step 0 (its stage is complete since this step's
            // barrier; after a tile's last step the values go unused)
#pragma unroll
            for (int x = 0; x < 4 * MI; ++x) {
                const int i = x >> 2, j = x & 3;
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1[i], b1[j], acc[i][j], 0, 0, 0);
                const int y = x - 2;
                if (y >= 0 && y < 4) b0[y] = opB(stn, 0, y);
                else if (y >= 4 && y < 4 + MI) a0[y - 4] = opA(stn, 0, y - 4);
            }
        }

        // 32x32 accumulator layout: lane holds column (lane & 31) and, in
        // register r, row 8 (r / 4) + 4 (lane / 32) + r % 4.
        const K2Tile tl = k2_decode(it * G + perm, tiles_m, tiles_n);
        const int ch = tl.ch, m0 = tl.m0, n0 = tl.n0;
        const int row0 = m0 + wm * 64 + 4 * hi, col0 = n0 + wn * 128 + rl;
        const bool full = m0 + BM <= M && n0 + BN <= N;
        if constexpr (CBLOCKED) {   // the sums (C included when accumulating) go straight out
            __amdgpu_buffer_rsrc_t rc[4];
            cdesc(tl, rc);
            const uint32_t vo = fresh(cvo);
#pragma unroll
            for (int x = 0; x < 4 * MI; ++x)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[x >> 2][x & 3][r]), rc[x & 3],
                                                          coff(vo, x, r), 0, 0);
            continue;
        }
        float* Cb = C + ch * sC + (int64_t)row0 * ldc + col0;
        const int64_t row_step = ldc;   // elements between rows
        // One 32 x 32 block at a time.  Accumulating, the block's 16 loads
        // go out together (a lane outside C reads C[0] instead) and are
        // waited for once, before its 16 guarded stores; element by element
        // the compiler would wait for every load.
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                float* pb = Cb + j * 32;   // column block j
                const bool colok = full || col0 + j * 32 < N;
                float v[16];
#pragma unroll
                for (int r = 0; r < 16; ++r) v[r] = acc[i][j][r];
                if (accumulate) {
                    float old[16];
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int dr = i * 32 + 8 * (r >> 2) + (r & 3);
                        const bool ok = colok && (full || row0 + dr < M);
                        old[r] = *(ok ? pb + (int64_t)dr * row_step : C);
                    }
#pragma unroll
                    for (int r = 0; r < 16; ++r) v[r] += old[r];
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int dr = i * 32 + 8 * (r >> 2) + (r & 3);
                    if (colok && (full || row0 + dr < M)) pb[(int64_t)dr * row_step] = v[r];
                }
            }
    }
}

// ---------------------------------------------------------------- fp32 VALU

template <bool BLOCKED>
__global__ __launch_bounds__(256) void k2_contract_f32(const float* __restrict__ A, const float* __restrict__ B,
                                                      float* __restrict__ C, int M, int N, int K, int64_t lda,
                                                      int64_t ldb, int64_t ldc, int64_t sA, int64_t sB,
                                                      int64_t sC, int accumulate,
                                                      const uint8_t* __restrict__ kmask) {
    __shared__ float As[16][64 + 4], Bs[16][64 + 4];
    const int64_t ch = blockIdx.z;
    const int m0 = blockIdx.x * 64, n0 = blockIdx.y * 64;
    const PanelGeom ga = panel_geom(M, K), gb = panel_geom(N, K);
    auto a_at = [&](int64_t r, int64_t k) { return BLOCKED ? A[panel_off(ga, ch, r, k)] : A[ch * sA + r * lda + k]; };
    auto b_at = [&](int64_t r, int64_t k) { return BLOCKED ? B[panel_off(gb, ch, r, k)] : B[ch * sB + r * ldb + k]; };
    float* Cr = C + ch * sC;
    const int t = threadIdx.x, tx = t & 15, ty = t >> 4;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int idx = t + 256 * s, row = idx >> 4, kk = idx & 15, k = k0 + kk;
            const bool kv = k < K && (!kmask || kmask[k] != 0);
            As[kk][row] = (m0 + row < M && kv) ? a_at(m0 + row, k) : 0.f;
            Bs[kk][row] = (n0 + row < N && kv) ? b_at(n0 + row, k) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 16; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                a[i] = As[kk][ty * 4 + i];
                b[i] = Bs[kk][tx * 4 + i];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] += a[i] * b[j];
        }
        __syncthreads();
    }
    const int64_t jblocks = (N + kResJ - 1) / kResJ;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int row = m0 + ty * 4 + i, col = n0 + tx * 4 + j;
            if (row < M && col < N) {
                float* p = BLOCKED ? C + result_off(jblocks, (int)gridDim.z, ch, row, col) : Cr + (int64_t)row * ldc + col;
                *p = accumulate ? *p + acc[i][j] : acc[i][j];
            }
        }
}

// Token mask of a tile's columns (0/1 bytes, zero from cols to cpad) followed
// by its rows (from byte cpad, zero from rows to rpad).
__global__ void k_stage_tile_mask(const uint8_t* __restrict__ mask, int64_t row0, int rows, int64_t col0, int cols,
                                  int cpad, int rpad, uint8_t* __restrict__ dst) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k < cpad) {
        dst[k] = (k < cols && (!mask || mask[col0 + k] != 0)) ? 1 : 0;
    } else if (k < cpad + rpad) {
        const int r = k - cpad;
        dst[k] = (r < rows && (!mask || mask[row0 + r] != 0)) ? 1 : 0;
    }
}

__global__ void k_stage_kmask(const uint8_t* __restrict__ mask, int klen, int padded, uint8_t* __restrict__ dst) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k < padded) dst[k] = (k < klen && (!mask || mask[k] != 0)) ? 1 : 0;
}

// Repack a device tile's row-major panel [ch][rows][ld] (bf16) into the
// blocked operand layout of the contraction, [ch][tiles][nk][256][32], with
// the staged k-mask applied and zeros for rows >= rows and k >= klen (the
// staged mask is 0 there).  One work-group per (two k-steps, 256-row tile,
// channel).  Thread t moves 16-byte piece e = t % 8 of the 128 bytes (two
// k-steps) of rows t / 8 + 32 j, j < 8: a load instruction reads eight whole
// 128-byte row segments, a store writes two runs of eight consecutive
// 64-byte block rows (one per k-step).
__global__ __launch_bounds__(256) void k_panel_block(const bf16_t* __restrict__ P, int rows, int ld, int64_t sP,
                                                     int tiles, int nk, const uint8_t* __restrict__ kst,
                                                     bf16_t* __restrict__ dst) {
    // Work-groups are dealt to the 8 XCDs round-robin by linear index; give
    // each XCD a contiguous run of (k-step pair, tile, channel) units, k-step
    // pairs fastest, so that the two 128-byte lines a row segment straddles
    // (rows are ld * 2 bytes apart, rarely a multiple of 128) are fetched
    // into one XCD's L2 and serve both neighbouring units.
    const unsigned gx = gridDim.x, gy = gridDim.y;
    const unsigned nu = gx * gy * gridDim.z, lin = blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z);
    const unsigned per = nu >> 3, extra = nu & 7, xcd = lin & 7;
    const unsigned u = xcd * per + min(xcd, extra) + (lin >> 3);   // a bijection of [0, nu)
    const int kp = (int)(u % gx), tile = (int)((u / gx) % gy), c = (int)(u / (gx * gy)), t = threadIdx.x;
    const int r0 = tile * 256;
    const int nrow = min(256, rows - r0);
    const int e = t & 7, h = e >> 2, q = e & 3;   // k-step 2 kp + h, k = 8 q .. + 7 within it
    const int kt = 2 * kp + h;
    // rows past the panel fall outside the descriptor and read as zero
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(P + c * sP + (int64_t)r0 * ld, (uint32_t)nrow * (uint32_t)ld * 2u);
    uint4 v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = buf_load16(rp, (uint32_t)(((t >> 3) + 32 * j) * ld + kp * 64 + 8 * e) * 2u);
    if (kt >= nk) return;   // the odd last k-step of the panel has no second half
    // staged 0/1 bytes of k = 32 kt + 8 q .. + 7 (fresh for every k < 32 nk)
    const uint2 m8 = *reinterpret_cast<const uint2*>(kst + kt * 32 + 8 * q);
    const uint32_t mw[2] = {m8.x, m8.y};
    uint32_t keep[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t b2 = mw[i >> 1] >> (16 * (i & 1));
        keep[i] = ((b2 & 0xffu) ? 0xffffu : 0u) | ((b2 & 0xff00u) ? 0xffff0000u : 0u);
    }
    bf16_t* out = dst + (((int64_t)c * tiles + tile) * nk + kt) * (256 * 32) + 8 * q;
#pragma unroll
    for (int j = 0; j < 8; ++j)
        *reinterpret_cast<uint4*>(out + ((t >> 3) + 32 * j) * 32) =
            make_uint4(v[j].x & keep[0], v[j].y & keep[1], v[j].z & keep[2], v[j].w & keep[3]);
}

}  // namespace

hipError_t launch_panel_block(const void* P, int64_t rows, int64_t ld, int64_t klen, int nch, const uint8_t* kst,
                              void* dst, hipStream_t s) {
    const int tiles = (int)((rows + 255) / 256), nk = (int)((klen + 31) / 32);
    hipLaunchKernelGGL(k_panel_block, dim3((unsigned)((nk + 1) / 2), (unsigned)tiles, (unsigned)nch), dim3(256), 0, s,
                       (const bf16_t*)P, (int)rows, (int)ld, rows * ld, tiles, nk, kst, (bf16_t*)dst);
    return hipGetLastError();
}

// The pair-blocked result is addressed per 64 rows of a column block with
// 32-bit byte offsets: 64 rows of jblocks * batch * 32 floats must stay
// below 4 GiB (N = 65536 with 128 channels uses half of it).
bool cblocked_fits(int64_t N, int batch) {
    const int64_t rs = (N + kResJ - 1) / kResJ * batch * kResJ;
    return 64 * rs * 4 < ((int64_t)1 << 32);
}

// Pacing needs whole XCD groups (G a multiple of 8, all resident) and at
// least two full rounds; it resets the counters first (a kernel, not a
// memset, so that the sequence can be captured in a graph).
namespace {
int pace_launch(int grid, int total, hipStream_t s) {
    if ((grid & 7) != 0 || total < 2 * grid) return 0;
    hipLaunchKernelGGL(k_pace_reset, dim3(1), dim3(8 * kPaceLine), 0, s);
    return 1;
}
}  // namespace

hipError_t launch_contract_blocked_rowc(const void* A, const void* B, float* C, int64_t M, int64_t N, int64_t K,
                                        int batch, int accumulate, int cus, hipStream_t s) {
    constexpr int BM = 256;
    const int tm = (int)((M + BM - 1) / BM), tn = (int)((N + BN - 1) / BN);
    const int total = tm * tn * batch;
    const int grid = total < cus ? total : cus;
    const int pace = pace_launch(grid, total, s);
    hipLaunchKernelGGL((k2_contract_ws<true, false, false>), dim3(grid), dim3(768), 0, s, (const bf16_t*)A,
                       (const bf16_t*)B, C, (int)M, (int)N, (int)K, 0, 0, N, (int64_t)0, (int64_t)0, M * N, tm, tn,
                       total, accumulate, (const uint8_t*)nullptr, pace);
    return hipGetLastError();
}

hipError_t launch_contract_blocked_packed(const void* A, const void* B, float* C, int64_t M, int64_t N, int64_t K,
                                          int batch, int accumulate, int cus, hipStream_t s) {
    constexpr int BM = 256;
    const int tm = (int)((M + BM - 1) / BM), tn = (int)((N + BN - 1) / BN);
    const int total = tm * tn * batch;
    const int grid = total < cus ? total : cus;
    if (!cblocked_fits(N, batch)) return hipErrorInvalidValue;
    const int pace = pace_launch(grid, total, s);
    hipLaunchKernelGGL((k2_contract_ws<true, false, true>), dim3(grid), dim3(768), 0, s, (const bf16_t*)A,
                       (const bf16_t*)B, C, (int)M, (int)N, (int)K, 0, 0, (int64_t)0, (int64_t)0, (int64_t)0,
                       (int64_t)0, tm, tn, total, accumulate, (const uint8_t*)nullptr, pace);
    return hipGetLastError();
}

hipError_t launch_contract_transposed(int ta, int tb, const void* A, const void* B, float* C, int64_t M, int64_t N,
                                      int64_t K, int batch, int cus, hipStream_t s, int accumulate) {
    constexpr int BM = 256;
    const int tm = (int)((M + BM - 1) / BM), tn = (int)((N + BN - 1) / BN);
    const int total = tm * tn * batch;
    const int grid = total < cus ? total : cus;
    if ((!ta && !tb) || !cblocked_fits(N, batch)) return hipErrorInvalidValue;
    const int pace = pace_launch(grid, total, s);
#define K2_TR(TA_, TB_)                                                                                             \
    hipLaunchKernelGGL((k2_contract_ws<true, false, true, TA_, TB_>), dim3(grid), dim3(768), 0, s, (const bf16_t*)A, \
                       (const bf16_t*)B, C, (int)M, (int)N, (int)K, 0, 0, (int64_t)0, (int64_t)0, (int64_t)0,     \
                       (int64_t)0, tm, tn, total, accumulate, (const uint8_t*)nullptr, pace)
    if (!ta && tb) K2_TR(false, true);
    else if (ta && tb) K2_TR(true, true);
    else K2_TR(true, false);
#undef K2_TR
    return hipGetLastError();
}

hipError_t launch_stage_tile_mask(const uint8_t* mask, int64_t row0, int64_t rows, int64_t col0, int64_t cols,
                                  uint8_t* dst, hipStream_t s) {
    const int cpad = (int)((cols + 31) / 32 * 32), rpad = (int)((rows + 3) / 4 * 4);
    hipLaunchKernelGGL(k_stage_tile_mask, dim3((unsigned)((cpad + rpad + 255) / 256)), dim3(256), 0, s, mask, row0,
                       (int)rows, col0, (int)cols, cpad, rpad, dst);
    return hipGetLastError();
}

hipError_t launch_stage_kmask(const uint8_t* mask, int64_t klen, uint8_t* dst, hipStream_t s) {
    const int padded = (int)((klen + 31) / 32 * 32);
    hipLaunchKernelGGL(k_stage_kmask, dim3((padded + 255) / 256), dim3(256), 0, s, mask, (int)klen, padded, dst);
    return hipGetLastError();
}

hipError_t launch_contract(int dtype, int blocked, const void* A, const void* B, float* C, int64_t M,
                           int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t ldc, int64_t sA,
                           int64_t sB, int64_t sC, int batch, int accumulate, const uint8_t* kmask, int cus,
                           hipStream_t s) {
    if (dtype == 0) {
        const dim3 grid((unsigned)((M + 63) / 64), (unsigned)((N + 63) / 64), (unsigned)batch);
        if (blocked)
            hipLaunchKernelGGL(k2_contract_f32<true>, grid, dim3(256), 0, s, (const float*)A, (const float*)B, C,
                               (int)M, (int)N, (int)K, lda, ldb, ldc, sA, sB, sC, accumulate, kmask);
        else
            hipLaunchKernelGGL(k2_contract_f32<false>, grid, dim3(256), 0, s, (const float*)A, (const float*)B, C,
                               (int)M, (int)N, (int)K, lda, ldb, ldc, sA, sB, sC, accumulate, kmask);
        return hipGetLastError();
    }
    constexpr int BM = 256;
    const int tm = (int)((M + BM - 1) / BM), tn = (int)((N + BN - 1) / BN);
    const int total = tm * tn * batch;
    const int grid = total < cus ? total : cus;
    const bf16_t* a = (const bf16_t*)A;
    const bf16_t* b = (const bf16_t*)B;
    if (blocked && !cblocked_fits(N, batch)) return hipErrorInvalidValue;
    const int pace = pace_launch(grid, total, s);
#define K2_WS(BL, KM)                                                                                              \
    hipLaunchKernelGGL((k2_contract_ws<BL, KM, BL>), dim3(grid), dim3(768), 0, s, a, b, C, (int)M, (int)N, (int)K, \
                       (int)lda, (int)ldb, ldc, sA, sB, sC, tm, tn, total, accumulate, kmask, pace)
    if (kmask) {
        if (blocked) K2_WS(true, true);
        else K2_WS(false, true);
    } else {
        if (blocked) K2_WS(true, false);
        else K2_WS(false, false);
    }
#undef K2_WS
    return hipGetLastError();
}

// Host-side walk over the direct-to-LDS loads of one k2_contract_ws launch,
// computed with the kernel's own addressing functions (k2_addr.h).
//
// Tile order: every (channel, row tile, column tile) must be taken by exactly
// one (work-group, round) of the persistent grid.  Loads: for the channels in
// `chans` (the kernel's addressing is the same in every channel apart from
// the channel offset, so the first and last channel bound it), every row tile
// of A and every column tile of B, every step, loader wave, load, lane and
// element: the descriptor must lie inside the operand's allocation (base >= 0,
// base + range <= bytes, range a multiple of 16), and every element the tile
// needs (row < rows, k < K) must be inside the range at the byte address the
// operand's layout gives it.  Elements the tile does not need (rows past the
// operand, k past K) may read anything inside the range, or zeros.
namespace {
int64_t k2_layout_off(const K2Operand& op, int ch, int64_t row, int64_t k) {
    if (op.mode == kK2Blocked) return panel_off(panel_geom(op.rows, op.K), ch, row, k);
    if (op.mode == kK2RowMajor) return (int64_t)ch * op.stride + row * op.ld + k;
    return panel_off(panel_geom(op.K, op.rows), ch, k, row);   // X[k][row] in the panel layout of X
}

void k2_check_operand(const K2Operand& op, uint64_t bytes, int ch, K2CheckCounts& n) {
    const int nk = (op.K + kK2BK - 1) / kK2BK;
    const int tiles = (op.rows + kK2Tile - 1) / kK2Tile;
    for (int tt = 0; tt < tiles; ++tt) {
        const int t0 = tt * kK2Tile;
        for (int kt = 0; kt < nk; ++kt) {
            const K2Desc d = k2_desc(op, ch, t0, kt);
            const bool desc_ok = d.base >= 0 && (d.range % 16) == 0 && (uint64_t)d.base * 2 + d.range <= bytes;
            for (int lw = 0; lw < kK2Loaders; ++lw)
                for (int jj = 0; jj < kK2LoadsPerOperand; ++jj) {
                    uint32_t off = 0;
                    const bool in = k2_load_off(op, t0, kt, lw, jj, off);
                    ++n.loads;
                    if (in && !desc_ok) ++n.bad_desc;
                    const uint32_t lds = k2_lds_off(lw, jj);
                    for (int lane = 0; lane < 64; ++lane) {
                        const uint64_t voff = (uint64_t)k2_lane_off(op, lw, lane) + off;
                        if (voff + 16 > 0xffffffffull) ++n.bad_elem;   // the lane offset is 32-bit
                        const uint32_t lb = lds + 16u * (uint32_t)lane;   // LDS byte the lane's 16 bytes go to
                        for (int e = 0; e < 8; ++e) {
                            int64_t row, k;
                            if (op.mode == kK2Transposed) {   // 2 KB per 32-column block, 64 bytes per k row
                                const int blk = (int)(lb / 2048), kr = (int)(lb % 2048) / kK2Row;
                                row = t0 + 32 * blk + ((lb % kK2Row) / 2 + e);
                                k = (int64_t)kt * kK2BK + kr;
                            } else {   // row r, slot s holds chunk s ^ ((r >> 2) & 3)
                                const int r = (int)(lb / kK2Row), slot = (int)(lb % kK2Row) / 16;
                                row = t0 + r;
                                k = (int64_t)kt * kK2BK + 8 * (slot ^ ((r >> 2) & 3)) + e;
                            }
                            if (row >= op.rows || k >= op.K) continue;   // not needed by the tile
                            ++n.elems;
                            const uint64_t byte = voff + 2u * (uint32_t)e;
                            const bool hit = in && byte + 2 <= d.range &&
                                             d.base * 2 + (int64_t)byte == 2 * k2_layout_off(op, ch, row, k);
                            if (!hit) ++n.bad_elem;
                        }
                    }
                }
        }
    }
}
}  // namespace

void k2_check_c(int64_t M, int64_t N, int batch, uint64_t c_bytes, int all_channels, K2CheckCounts& n) {
    n = K2CheckCounts{};
    const int tm = (int)((M + kK2Tile - 1) / kK2Tile), tn = (int)((N + kK2Tile - 1) / kK2Tile);
    const int J = (int)((N + kResJ - 1) / kResJ);
    const uint32_t crs = k2_c_row_floats((int)N, batch);
    n.tiles = (int64_t)tm * tn * batch;
    for (int ch = 0; ch < batch; ++ch) {
        if (!all_channels && ch != 0 && ch != batch - 1) continue;
        std::vector<uint8_t> hit((size_t)M * (size_t)N, 0);
        for (int ti = 0; ti < tm; ++ti)
            for (int tj = 0; tj < tn; ++tj) {
                const K2Tile t{ch, ti * kK2Tile, tj * kK2Tile};
                for (int wave = 0; wave < 8; ++wave)
                    for (int j = 0; j < 4; ++j) {
                        const K2Desc d = k2_c_desc((int)M, (int)N, batch, t, wave, j);
                        if (d.range && (d.base < 0 || (uint64_t)d.base * 4 + d.range > c_bytes)) ++n.bad_desc;
                        for (int xr = 0; xr < 2; ++xr) {
                            const int x = 4 * xr + j;
                            ++n.loads;
                            for (int r = 0; r < 16; ++r)
                                for (int lane = 0; lane < 64; ++lane) {
                                    int row, col;
                                    k2_c_elem(t, wave, lane, x, r, row, col);
                                    const uint64_t off = (uint64_t)k2_c_lane_off(crs, lane) + k2_c_reg_off(crs, x, r);
                                    const bool in = off < d.range;
                                    if (!in) {   // must be a row past M or a column block past C's last
                                        if (row < M && col / kResJ < J) ++n.bad_elem;
                                        continue;
                                    }
                                    // accessed: the element the layout puts there, inside C
                                    const int64_t want = result_off(J, batch, ch, row, col);
                                    if (off % 4 || d.base + (int64_t)(off / 4) != want || row >= M || col / kResJ >= J)
                                        ++n.bad_elem;
                                    if (row < M && col < N) {
                                        ++n.elems;
                                        uint8_t& h = hit[(size_t)row * N + col];
                                        if (h) ++n.bad_elem;
                                        h = 1;
                                    }
                                }
                        }
                    }
            }
        for (uint8_t h : hit) n.bad_elem += h ? 0 : 1;
    }
}

void k2_check_loads(int a_mode, int b_mode, int64_t M, int64_t N, int64_t K, int64_t lda, int64_t ldb, int64_t sA,
                    int64_t sB, int batch, uint64_t a_bytes, uint64_t b_bytes, int grid, int all_channels,
                    K2CheckCounts& n) {
    n = K2CheckCounts{};
    const int tm = (int)((M + kK2Tile - 1) / kK2Tile), tn = (int)((N + kK2Tile - 1) / kK2Tile);
    const int64_t total = (int64_t)tm * tn * batch;
    std::vector<uint8_t> seen((size_t)total, 0);
    for (int wg = 0; wg < grid; ++wg) {
        const int perm = k2_perm(wg, grid), mine = k2_my_tiles(perm, grid, (int)total);
        for (int it = 0; it < mine; ++it) {
            const K2Tile t = k2_decode(it * grid + perm, tm, tn);
            const bool ok = t.ch >= 0 && t.ch < batch && t.m0 >= 0 && t.m0 < M && t.n0 >= 0 && t.n0 < N &&
                            t.m0 % kK2Tile == 0 && t.n0 % kK2Tile == 0;
            if (!ok) {
                ++n.bad_tiles;
                continue;
            }
            uint8_t& v = seen[((size_t)t.ch * tm + t.m0 / kK2Tile) * tn + t.n0 / kK2Tile];
            if (v) ++n.bad_tiles;
            v = 1;
        }
    }
    for (uint8_t v : seen) n.bad_tiles += v ? 0 : 1;
    n.tiles = total;
    const K2Operand opa{a_mode, (int)M, (int)K, (int)lda, sA}, opb{b_mode, (int)N, (int)K, (int)ldb, sB};
    for (int ch = 0; ch < batch; ++ch) {
        if (!all_channels && ch != 0 && ch != batch - 1) continue;
        k2_check_operand(opa, a_bytes, ch, n);
        k2_check_operand(opb, b_bytes, ch, n);
    }
}

}  // namespace trimul
