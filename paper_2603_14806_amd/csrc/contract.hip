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
#include "common.h"
#include "kernels.h"

namespace trimul {
namespace {

// ---------------------------------------------------------------- bf16 MFMA
//
// Macro tile 256 x 256, k-tile 64, 256 threads = 4 waves in a 2 x 2 grid,
// each wave owns a 128 x 128 sub-tile = 4 x 4 MFMA blocks of 32 x 32.
// Two LDS stages of (A 256x64 + B 256x64) bf16 = 128 KB.  Each LDS row holds
// 64 k-values = 8 chunks of 16 bytes; chunk q of row r is stored at slot
// q ^ (r & 7) so that the 32 rows a wave reads at one k-chunk hit distinct
// banks.
constexpr int BM = 256, BN = 256, BK = 64;
constexpr int ROW_BYTES = BK * 2;               // 128
constexpr int A_BYTES = BM * ROW_BYTES;         // 32 KB
constexpr int B_BYTES = BN * ROW_BYTES;         // 32 KB
constexpr int STAGE_BYTES = A_BYTES + B_BYTES;  // 64 KB

__device__ __forceinline__ uint32_t lane_keep(bool v) { return v ? 0xffffu : 0u; }

// Zero the bf16 elements of a 16-byte chunk whose k (k_base + e) is >= K or,
// with a token mask, masked out.
template <bool KMASK>
__device__ __forceinline__ uint4 chunk_keep_mask(int k_base, int K, const uint8_t* __restrict__ kmask) {
    uint32_t m[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        const int k = k_base + 2 * h;
        bool v0 = k < K, v1 = k + 1 < K;
        if (KMASK) {
            v0 = v0 && kmask[k] != 0;
            v1 = v1 && kmask[k + 1] != 0;
        }
        m[h] = lane_keep(v0) | (lane_keep(v1) << 16);
    }
    return make_uint4(m[0], m[1], m[2], m[3]);
}

__device__ __forceinline__ uint4 and4(uint4 a, uint4 b) {
    return make_uint4(a.x & b.x, a.y & b.y, a.z & b.z, a.w & b.w);
}

template <bool KMASK>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))
void k2_contract_mfma(const bf16_t* __restrict__ A, const bf16_t* __restrict__ B, float* __restrict__ C,
                      int M, int N, int K, int lda, int ldb, int64_t ldc, int64_t sA, int64_t sB,
                      int64_t sC, int tiles_m, int tiles_n, int total, int accumulate,
                      const uint8_t* __restrict__ kmask) {
    __shared__ __attribute__((aligned(16))) char smem[2 * STAGE_BYTES];

    // Work-group -> tile.  Work-groups are dealt round-robin to the 8 XCDs;
    // give each XCD a contiguous range of logical tiles so that the tiles
    // sharing A row-panels and B column-panels meet in the same L2.
    const int bid = blockIdx.x;
    const int per = total >> 3;
    const int logical = bid < (per << 3) ? (bid & 7) * per + (bid >> 3) : bid;
    const int tiles = tiles_m * tiles_n;
    const int ch = logical / tiles;
    const int rem = logical - ch * tiles;
    constexpr int G = 4;   // tile rows per group: 4 x tiles_n tiles walk down 4 A row-panels
    const int gid = rem / (G * tiles_n);
    const int first_m = gid * G;
    const int gsz = min(tiles_m - first_m, G);
    const int in_g = rem - gid * G * tiles_n;
    const int tm = first_m + in_g % gsz;
    const int tn = in_g / gsz;
    const int m0 = tm * BM, n0 = tn * BN;

    const bf16_t* Ab = A + ch * sA + (int64_t)m0 * lda;
    const bf16_t* Bb = B + ch * sB + (int64_t)n0 * ldb;
    // Rows past M (N) fall outside the resource and load as zero.
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(Ab, (uint32_t)(min(BM, M - m0) * lda * 2));
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(Bb, (uint32_t)(min(BN, N - n0) * ldb * 2));

    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int wm = wave >> 1, wn = wave & 1;

    // Global -> LDS copy: thread t moves chunk kc = t & 7 of rows (t >> 3) + 32 s.
    const int row_l = t >> 3, kc = t & 7;
    const uint32_t ga_off = (uint32_t)(row_l * lda + kc * 8) * 2;
    const uint32_t gb_off = (uint32_t)(row_l * ldb + kc * 8) * 2;
    const uint32_t ga_step = (uint32_t)(32 * lda * 2), gb_step = (uint32_t)(32 * ldb * 2);
    const uint32_t lds_w = row_l * ROW_BYTES + ((kc ^ (row_l & 7)) << 4);

    // LDS -> MFMA operands: lane reads row (lane & 31) of its 32-row block at
    // k-chunk 2 s + (lane >> 5) of the k-tile.
    uint32_t a_rd[4], b_rd[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const uint32_t x = ((2 * s + (lane >> 5)) ^ (lane & 7)) << 4;
        a_rd[s] = (wm * 128 + (lane & 31)) * ROW_BYTES + x;
        b_rd[s] = A_BYTES + (wn * 128 + (lane & 31)) * ROW_BYTES + x;
    }

    f32x16_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    uint4 sa[8], sb[8];
    const int nk = (K + BK - 1) / BK;

    auto gload = [&](int kt) {
        const uint32_t kb = (uint32_t)kt * ROW_BYTES;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            sa[s] = buf_load16(ra, ga_off + s * ga_step + kb);
            sb[s] = buf_load16(rb, gb_off + s * gb_step + kb);
        }
        if (KMASK || kt * BK + BK > K) {
            const uint4 keep = chunk_keep_mask<KMASK>(kt * BK + kc * 8, K, kmask);
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                sa[s] = and4(sa[s], keep);
                sb[s] = and4(sb[s], keep);
            }
        }
    };
    auto lstore = [&](int stage) {
        char* base = smem + stage * STAGE_BYTES + lds_w;
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            *reinterpret_cast<uint4*>(base + s * 32 * ROW_BYTES) = sa[s];
            *reinterpret_cast<uint4*>(base + A_BYTES + s * 32 * ROW_BYTES) = sb[s];
        }
    };

    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt & 1;
        if (kt + 1 < nk) gload(kt + 1);
        const char* st = smem + cur * STAGE_BYTES;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            bf16x8_t af[4], bfr[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const bf16x8_t*>(st + a_rd[s] + i * 32 * ROW_BYTES);
#pragma unroll
            for (int j = 0; j < 4; ++j) bfr[j] = *reinterpret_cast<const bf16x8_t*>(st + b_rd[s] + j * 32 * ROW_BYTES);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) lstore(cur ^ 1);
        __syncthreads();
    }

    // 32x32 accumulator layout: lane holds column (lane & 31) and, in register
    // r, row 8 (r / 4) + 4 (lane / 32) + r % 4.
    float* Cb = C + ch * sC;
    const int lrow = 4 * (lane >> 5), lcol = lane & 31;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int col = n0 + wn * 128 + j * 32 + lcol;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm * 128 + i * 32 + 8 * (r >> 2) + lrow + (r & 3);
                if (row < M && col < N) {
                    float* p = Cb + (int64_t)row * ldc + col;
                    float v = acc[i][j][r];
                    if (accumulate) v += *p;
                    *p = v;
                }
            }
        }
}

// ---------------------------------------------------------------- fp32 VALU

__global__ __launch_bounds__(256) void k2_contract_f32(const float* __restrict__ A, const float* __restrict__ B,
                                                      float* __restrict__ C, int M, int N, int K, int64_t lda,
                                                      int64_t ldb, int64_t ldc, int64_t sA, int64_t sB,
                                                      int64_t sC, int accumulate,
                                                      const uint8_t* __restrict__ kmask) {
    __shared__ float As[16][64 + 4], Bs[16][64 + 4];
    const int64_t ch = blockIdx.z;
    const int m0 = blockIdx.x * 64, n0 = blockIdx.y * 64;
    A += ch * sA;
    B += ch * sB;
    C += ch * sC;
    const int t = threadIdx.x, tx = t & 15, ty = t >> 4;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int idx = t + 256 * s, row = idx >> 4, kk = idx & 15, k = k0 + kk;
            const bool kv = k < K && (!kmask || kmask[k] != 0);
            As[kk][row] = (m0 + row < M && kv) ? A[(int64_t)(m0 + row) * lda + k] : 0.f;
            Bs[kk][row] = (n0 + row < N && kv) ? B[(int64_t)(n0 + row) * ldb + k] : 0.f;
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
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int row = m0 + ty * 4 + i, col = n0 + tx * 4 + j;
            if (row < M && col < N) {
                float* p = C + (int64_t)row * ldc + col;
                *p = accumulate ? *p + acc[i][j] : acc[i][j];
            }
        }
}

}  // namespace

hipError_t launch_contract(int dtype, const void* A, const void* B, float* C, int64_t M, int64_t N,
                           int64_t K, int64_t lda, int64_t ldb, int64_t ldc, int64_t sA, int64_t sB,
                           int64_t sC, int batch, int accumulate, const uint8_t* kmask,
                           hipStream_t s) {
    if (dtype == 0) {
        const dim3 grid((unsigned)((M + 63) / 64), (unsigned)((N + 63) / 64), (unsigned)batch);
        hipLaunchKernelGGL(k2_contract_f32, grid, dim3(256), 0, s, (const float*)A, (const float*)B, C, (int)M,
                           (int)N, (int)K, lda, ldb, ldc, sA, sB, sC, accumulate, kmask);
        return hipGetLastError();
    }
    const int tm = (int)((M + BM - 1) / BM), tn = (int)((N + BN - 1) / BN);
    const int total = tm * tn * batch;
    if (kmask)
        hipLaunchKernelGGL((k2_contract_mfma<true>), dim3(total), dim3(256), 0, s, (const bf16_t*)A,
                           (const bf16_t*)B, C, (int)M, (int)N, (int)K, (int)lda, (int)ldb, ldc, sA, sB, sC,
                           tm, tn, total, accumulate, kmask);
    else
        hipLaunchKernelGGL((k2_contract_mfma<false>), dim3(total), dim3(256), 0, s, (const bf16_t*)A,
                           (const bf16_t*)B, C, (int)M, (int)N, (int)K, (int)lda, (int)ldb, ldc, sA, sB, sC,
                           tm, tn, total, accumulate, kmask);
    return hipGetLastError();
}

}  // namespace trimul
