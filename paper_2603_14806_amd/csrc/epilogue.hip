// K3: output LayerNorm over the hidden channels, output projection, sigmoid
// gate recomputed from LN_in(z), and pair mask (the gated output of the
// triangle update, Section 3.3).  Reads the channel-major fp32 contraction
// result and writes the pair-major update [rows][cols][c_z].
//
// Work unit: 64 consecutive pairs of one output row.
#include "common.h"
#include "kernels.h"

namespace trimul {
namespace {

constexpr int kPairs = 64;

template <typename T, typename TO>
__global__ __launch_bounds__(256) void k3_epilogue_valu(
    EpilogueArgs a, int64_t nchunk, const float* __restrict__ wo_t, const float* __restrict__ wg_t,
    const float* __restrict__ lnin_w, const float* __restrict__ lnin_b,
    const float* __restrict__ lnout_w, const float* __restrict__ lnout_b, float eps) {
    __shared__ float cs[kPairs][kCh + 1];
    __shared__ float xs[kPairs][kCz + 1];
    const int t = threadIdx.x;
    const int64_t i = blockIdx.x / nchunk;
    const int64_t j0 = (blockIdx.x % nchunk) * kPairs;
    const int np = (int)min<int64_t>(kPairs, a.cols - j0);
    const T* z = static_cast<const T*>(a.z);

    const int64_t jblocks = (a.cols + kResJ - 1) / kResJ;
    for (int idx = t; idx < kPairs * kCh; idx += 256) {
        const int c = idx / kPairs, p = idx % kPairs;
        cs[p][c] = p < np ? (a.cblocked ? a.C[result_off(jblocks, kCh, c, i, j0 + p)] : a.C[c * a.sc + i * a.ldc + j0 + p])
                          : 0.f;
    }
    for (int idx = t; idx < kPairs * kCz; idx += 256) {
        const int p = idx / kCz, d = idx % kCz;
        xs[p][d] = p < np ? Store<T>::ld(z + ((i * a.cols) + j0 + p) * kCz + d) : 0.f;
    }
    __syncthreads();

    {   // both LayerNorms, four lanes per pair
        const int p = t >> 2, q = t & 3;
        float s1 = 0.f, s2 = 0.f;
        for (int d = q * 32; d < q * 32 + 32; ++d) {
            s1 += cs[p][d];
            s2 += xs[p][d];
        }
        s1 = sum_lanes4(s1);
        s2 = sum_lanes4(s2);
        const float mu1 = s1 * (1.0f / kCh), mu2 = s2 * (1.0f / kCz);
        float v1 = 0.f, v2 = 0.f;
        for (int d = q * 32; d < q * 32 + 32; ++d) {
            const float e1 = cs[p][d] - mu1, e2 = xs[p][d] - mu2;
            v1 += e1 * e1;
            v2 += e2 * e2;
        }
        v1 = sum_lanes4(v1);
        v2 = sum_lanes4(v2);
        const float r1 = rsqrtf(v1 * (1.0f / kCh) + eps), r2 = rsqrtf(v2 * (1.0f / kCz) + eps);
        for (int d = q * 32; d < q * 32 + 32; ++d) {
            cs[p][d] = (cs[p][d] - mu1) * r1 * lnout_w[d] + lnout_b[d];
            xs[p][d] = (xs[p][d] - mu2) * r2 * lnin_w[d] + lnin_b[d];
        }
    }
    __syncthreads();

    const int d = t & (kCz - 1), half = t >> 7;
    float y[32], gl[32];
#pragma unroll
    for (int q = 0; q < 32; ++q) y[q] = gl[q] = 0.f;
    for (int c = 0; c < kCh; ++c) {
        const float w = wo_t[c * kCz + d];
#pragma unroll
        for (int q = 0; q < 32; ++q) y[q] += w * cs[half * 32 + q][c];
    }
    for (int e = 0; e < kCz; ++e) {
        const float w = wg_t[e * kCz + d];
#pragma unroll
        for (int q = 0; q < 32; ++q) gl[q] += w * xs[half * 32 + q][e];
    }
    const bool mi = a.mask ? a.mask[a.row0 + i] != 0 : true;
    TO* out = static_cast<TO*>(a.out);
#pragma unroll
    for (int q = 0; q < 32; ++q) {
        const int p = half * 32 + q;
        if (p < np) {
            const bool m = mi && (a.mask ? a.mask[a.col0 + j0 + p] != 0 : true);
            Store<TO>::st(out + ((i * a.cols) + j0 + p) * kCz + d, m ? sigmoidf_(gl[q]) * y[q] : 0.f);
        }
    }
}


// ------------------------------------------------------------ bf16 MFMA
//
// Persistent kernel, 4 waves, work unit = 32 consecutive pairs of one output
// row.  Wave w owns output channels [32 w, 32 w + 32) of both W_o and W_g,
// kept in VGPRs as the MFMA B operand; the activations (LN_out(C) split into
// bf16 hi + lo, and bf16 LN_in(z) for the gate) are the A operand, so a lane
// ends up holding 32 consecutive output channels of a pair and the stores are
// 128-byte rows.
constexpr int kP3 = 32;
constexpr int kCsRow = kP3 + 4;     // C staging row stride (floats): conflict-free column reads
constexpr int kYRow = 256;          // bytes of one bf16 activation row [128]
constexpr int kOsRow = kCz + 8;     // output staging row stride (floats): the two half-waves hit disjoint banks

__device__ __forceinline__ uint32_t yoff(int p, int chunk) {
    return (uint32_t)(p * kYRow + ((chunk ^ (p & 15)) << 4));
}

template <typename TO, bool VEC_C, bool CBLK>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(2, 2)))
void k3_epilogue_mfma(EpilogueArgs a, int nchunk, int64_t nunits, const bf16_t* __restrict__ wepi,
                      const float* __restrict__ lnin_w, const float* __restrict__ lnin_b,
                      const float* __restrict__ lnout_w, const float* __restrict__ lnout_b, float eps) {
    __shared__ __attribute__((aligned(16))) float cs[kCh * kCsRow];          // C as [c][p]
    __shared__ __attribute__((aligned(16))) char ys[3][kP3 * kYRow];         // y_hi, y_lo, x_hi
    __shared__ __attribute__((aligned(16))) float prm[4][128];               // LN gains and biases
    __shared__ __attribute__((aligned(16))) float os[kP3 * kOsRow];          // outputs as [p][d]
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int lp = t >> 3, lq = t & 7;     // LayerNorms: pair lp, 8 lanes per pair
    const bf16_t* z = static_cast<const bf16_t*>(a.z);
    TO* out = static_cast<TO*>(a.out);

    bf16x8_t wo[8], wg[8];
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
        const size_t col = (size_t)ks * 16 + 8 * (lane >> 5);
        wo[ks] = *reinterpret_cast<const bf16x8_t*>(wepi + (size_t)(w * 32 + (lane & 31)) * 128 + col);
        wg[ks] = *reinterpret_cast<const bf16x8_t*>(wepi + (size_t)(128 + w * 32 + (lane & 31)) * 128 + col);
    }
    if (t < 128) {
        prm[0][t] = lnout_w[t];
        prm[1][t] = lnout_b[t];
        prm[2][t] = lnin_w[t];
        prm[3][t] = lnin_b[t];
    }

    // C loads: thread moves floats [4 cj, 4 cj + 4) of channel rows (t >> 3) + 32 s.
    const int cj = t & 7;
    auto load_c = [&](int64_t u, float4 (&cv)[4], uint4& z0, uint4& z1) {
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) cv[s2] = make_float4(0.f, 0.f, 0.f, 0.f);
        z0 = z1 = make_uint4(0, 0, 0, 0);
        if (u >= nunits) return;
        const uint32_t uq = (uint32_t)u / (uint32_t)nchunk;   // units < 2^31
        const int64_t i = uq, j0 = (int64_t)((uint32_t)u - uq * (uint32_t)nchunk) * kP3;
        const int np = (int)min<int64_t>(kP3, a.cols - j0);
        if (CBLK) {   // the unit's 128 channels x 32 pairs are one contiguous block
            const float4* blk = reinterpret_cast<const float4*>(a.C + result_off(nchunk, kCh, 0, i, j0));
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) {
                float4 v = blk[t + 256 * s2];
                if (4 * cj + 4 > np) {   // pairs past the end of the row are padding
                    if (4 * cj + 0 >= np) v.x = 0.f;
                    if (4 * cj + 1 >= np) v.y = 0.f;
                    if (4 * cj + 2 >= np) v.z = 0.f;
                    if (4 * cj + 3 >= np) v.w = 0.f;
                }
                cv[s2] = v;
            }
        }
#pragma unroll
        for (int s2 = 0; s2 < 4 && !CBLK; ++s2) {
            const float* src = a.C + (int64_t)((t >> 3) + 32 * s2) * a.sc + i * a.ldc + j0 + 4 * cj;
            if (VEC_C && 4 * cj + 4 <= np) {
                cv[s2] = *reinterpret_cast<const float4*>(src);
            } else {
                float e[4] = {0.f, 0.f, 0.f, 0.f};
                for (int k = 0; k < 4; ++k)
                    if (4 * cj + k < np) e[k] = src[k];
                cv[s2] = make_float4(e[0], e[1], e[2], e[3]);
            }
        }
        if (lp < np) {
            const uint4* zs = reinterpret_cast<const uint4*>(z + ((i * a.cols) + j0 + lp) * kCz + 16 * lq);
            z0 = zs[0];
            z1 = zs[1];
        }
    };

    float4 cc[4];
    uint4 zc0, zc1;
    load_c(blockIdx.x, cc, zc0, zc1);
    for (int64_t u = blockIdx.x; u < nunits; u += gridDim.x) {
        float4 cn[4];
        uint4 zn0, zn1;
        load_c(u + gridDim.x, cn, zn0, zn1);      // prefetch the next unit

#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2)
            *reinterpret_cast<float4*>(&cs[((t >> 3) + 32 * s2) * kCsRow + 4 * cj]) = cc[s2];
        __syncthreads();

        {   // LN_out over the 128 hidden channels of pair lp: lane lq holds c = lq + 8 i
            float v[16];
            float s1 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                v[i] = cs[(lq + 8 * i) * kCsRow + lp];
                s1 += v[i];
            }
            s1 = sum_lanes8(s1);
            const float mu = s1 * (1.0f / kCh);
            float q2 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                v[i] -= mu;
                q2 += v[i] * v[i];
            }
            q2 = sum_lanes8(q2);
            const float rs = rsqrtf(q2 * (1.0f / kCh) + eps);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int c = lq + 8 * i;
                const float y = v[i] * rs * prm[0][c] + prm[1][c];
                const bf16_t h = f2bf(y);
                const uint32_t o = yoff(lp, c >> 3) + 2 * (c & 7);
                *reinterpret_cast<bf16_t*>(ys[0] + o) = h;
                *reinterpret_cast<bf16_t*>(ys[1] + o) = f2bf(y - bf2f(h));
            }
        }
        {   // LN_in over the 128 pair channels of pair lp: lane lq holds 16 lq .. 16 lq + 15
            float v[16];
            const uint32_t uu[8] = {zc0.x, zc0.y, zc0.z, zc0.w, zc1.x, zc1.y, zc1.z, zc1.w};
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                v[2 * i] = __uint_as_float(uu[i] << 16);
                v[2 * i + 1] = __uint_as_float(uu[i] & 0xffff0000u);
            }
            float s1 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) s1 += v[i];
            s1 = sum_lanes8(s1);
            const float mu = s1 * (1.0f / kCz);
            float q2 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                v[i] -= mu;
                q2 += v[i] * v[i];
            }
            q2 = sum_lanes8(q2);
            const float rs = rsqrtf(q2 * (1.0f / kCz) + eps);
            uint32_t hx[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int c = 16 * lq + 2 * i;
                const float x0 = v[2 * i] * rs * prm[2][c] + prm[3][c];
                const float x1 = v[2 * i + 1] * rs * prm[2][c + 1] + prm[3][c + 1];
                hx[i] = (uint32_t)f2bf(x0) | ((uint32_t)f2bf(x1) << 16);
            }
            *reinterpret_cast<uint4*>(ys[2] + yoff(lp, 2 * lq)) = make_uint4(hx[0], hx[1], hx[2], hx[3]);
            *reinterpret_cast<uint4*>(ys[2] + yoff(lp, 2 * lq + 1)) = make_uint4(hx[4], hx[5], hx[6], hx[7]);
        }
        __syncthreads();

        f32x16_t ay, ag;
#pragma unroll
        for (int r = 0; r < 16; ++r) ay[r] = ag[r] = 0.f;
        const int ap = lane & 31;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            const uint32_t o = yoff(ap, 2 * ks + (lane >> 5));
            const bf16x8_t yh = *reinterpret_cast<const bf16x8_t*>(ys[0] + o);
            const bf16x8_t yl = *reinterpret_cast<const bf16x8_t*>(ys[1] + o);
            const bf16x8_t xh = *reinterpret_cast<const bf16x8_t*>(ys[2] + o);
            ay = __builtin_amdgcn_mfma_f32_32x32x16_bf16(yh, wo[ks], ay, 0, 0, 0);
            ag = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xh, wg[ks], ag, 0, 0, 0);
            ay = __builtin_amdgcn_mfma_f32_32x32x16_bf16(yl, wo[ks], ay, 0, 0, 0);
        }

        // Lane holds output channel 32 w + (lane & 31); register r holds pair
        // 8 (r / 4) + 4 (lane / 32) + r % 4.  Stage the unit's outputs in LDS,
        // then write its contiguous [32 pairs][128] block with 16-byte stores.
        const uint32_t uq = (uint32_t)u / (uint32_t)nchunk;   // units < 2^31
        const int64_t i = uq, j0 = (int64_t)((uint32_t)u - uq * (uint32_t)nchunk) * kP3;
        const int np = (int)min<int64_t>(kP3, a.cols - j0);
        const bool mi = a.mask ? a.mask[a.row0 + i] != 0 : true;
        const int d = w * 32 + (lane & 31);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int p = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            const bool m = p < np && mi && (a.mask ? a.mask[a.col0 + j0 + p] != 0 : true);
            os[p * kOsRow + d] = m ? sigmoidf_(ag[r]) * ay[r] : 0.f;
        }
        __syncthreads();
        TO* ob = out + ((i * a.cols) + j0) * kCz;
        const bool full = np == kP3;   // uniform: no per-lane predicates on full units
        if (sizeof(TO) == 4) {
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) {
                const int q = t + 256 * s2, p = q >> 5, d4 = (q & 31) * 4;
                if (full || p < np)
                    *reinterpret_cast<float4*>(reinterpret_cast<float*>(ob) + p * kCz + d4) =
                        *reinterpret_cast<const float4*>(&os[p * kOsRow + d4]);
            }
        } else {
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                const int q = t + 256 * s2, p = q >> 4, d8 = (q & 15) * 8;
                if (full || p < np) {
                    const float4 f0 = *reinterpret_cast<const float4*>(&os[p * kOsRow + d8]);
                    const float4 f1 = *reinterpret_cast<const float4*>(&os[p * kOsRow + d8 + 4]);
                    uint4 pk;
                    pk.x = (uint32_t)f2bf(f0.x) | ((uint32_t)f2bf(f0.y) << 16);
                    pk.y = (uint32_t)f2bf(f0.z) | ((uint32_t)f2bf(f0.w) << 16);
                    pk.z = (uint32_t)f2bf(f1.x) | ((uint32_t)f2bf(f1.y) << 16);
                    pk.w = (uint32_t)f2bf(f1.z) | ((uint32_t)f2bf(f1.w) << 16);
                    *reinterpret_cast<uint4*>(reinterpret_cast<bf16_t*>(ob) + p * kCz + d8) = pk;
                }
            }
        }
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) cc[s2] = cn[s2];
        zc0 = zn0;
        zc1 = zn1;
    }
}

// ---------------------------------------------------------------- ring variant
//
// The full update's epilogue (C in the pair-blocked layout, z [N][N][c_z]).
// Same work split and arithmetic as k3_epilogue_mfma, but C, z and the mask
// bytes of later units arrive by direct-to-LDS loads into a ring (three
// stages, two units ahead, with fp32 output; two with bf16 output, whose
// staging takes the room) while the current unit is computed, and the bf16
// activations are written back into the stage they were read from.  Masked
// pairs get y = LN_out(C) = 0, so their outputs are exactly 0 without a
// mask in the gating.  Every wave issues 7 loads and a fixed number of
// range-checked buffer stores per unit (tail pairs are dropped by the range
// check), so the vmcnt waits are constants.
//
// Stage layout (bytes):
//   [0, 16384)      C of the unit, [128 channels][32 pairs] fp32: chunk q
//                   (pairs 4q .. 4q + 3) of channel row c at slot q ^ h(c),
//                   h(c) = (c + c / 16) % 8, so that the 8 lanes reading
//                   channels 16 l + k (l = 0..7) of one pair hit 8 slots;
//                   afterwards y_hi [0, 8192) and y_lo [8192, 16384)
//   [16384, 24576)  z of the unit, [32 pairs][128] bf16: chunk q of pair row p
//                   at slot q ^ (p & 1); afterwards x_hi
//   [24576, 25600)  per-wave mask bytes: column mask bytes j0 .. j0 + 31 at 0,
//                   the dword of row mask byte i at 32 (0/1 bytes staged by
//                   launch_stage_tile_mask: columns, zero past cols, then rows
//                   from byte rmoff)
constexpr int kRC = 16384, kRZ = 8192, kRM = 1024;
constexpr int kRSt = kRC + kRZ + kRM;

template <typename TO>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(2, 2)))
void k3_epilogue_ring(const float* __restrict__ C, const bf16_t* __restrict__ z, const uint8_t* __restrict__ tmask,
                      int rows, int cols, int rmoff, int nunits, TO* __restrict__ out, const bf16_t* __restrict__ wepi,
                      const float* __restrict__ lnin_w, const float* __restrict__ lnin_b,
                      const float* __restrict__ lnout_w, const float* __restrict__ lnout_b, float eps) {
    // fp32 output leaves straight from the accumulators (a register holds 32
    // consecutive channels of one pair per half-wave: two whole 128-byte
    // rows per store), which frees the output staging for a third ring
    // stage; bf16 output is staged as [p][d] for 16-byte stores.
    constexpr bool kDirect = sizeof(TO) == 4;
    constexpr int kStages = kDirect ? 3 : 2;
    __shared__ __attribute__((aligned(16))) char ring[kStages * kRSt];
    // LN gains and biases; channel c at (c / 16) * 20 + c % 16, so that the 8
    // broadcast addresses of a read (c = 16 lq + 2 k) fall in distinct banks
    __shared__ __attribute__((aligned(16))) float prm[4][8 * 20];
    __shared__ __attribute__((aligned(16))) float os[kDirect ? 4 : kP3 * kOsRow];   // outputs as [p][d]
    const int t = threadIdx.x, lane = t & 63;
    const int w = __builtin_amdgcn_readfirstlane(t >> 6);
    const int lp = t >> 3, lq = t & 7;     // LayerNorms: pair lp, 8 lanes per pair
    const int G = gridDim.x;
    const int first = (G & 7) == 0 ? (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3) : blockIdx.x;
    const int nchunk = (cols + kP3 - 1) / kP3;
    constexpr int kStores = (int)(kP3 * kCz * sizeof(TO)) / (4 * 1024);   // staged path: 16-byte stores per lane
    constexpr int kS = kDirect ? 16 : kStores;                             // stores per lane per unit

    // Ring fill.  C: load k of wave w covers channel rows c = 8 (4 w + k) .. + 7,
    // lane -> row c + lane / 8 at slot lane % 8, which holds chunk
    // (lane % 8) ^ h(c) (h(c) = (lane / 8 + 2 w + k / 2) % 8 for these rows).
    // z and mask as in the projection.
    const uint32_t ring_base = lds_addr(ring);
    uint32_t cvo[2];
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
        cvo[kh] = (uint32_t)((lane >> 3) * 128 + (((lane & 7) ^ (((lane >> 3) + 2 * w + kh) & 7)) << 4)) +
                  (uint32_t)w * 4096;
    const int drow = w * 8 + (lane >> 4);
    const uint32_t dchunk = (uint32_t)(((lane & 15) ^ (drow & 1)) << 4);
    const uint32_t dv0 = (uint32_t)drow * kYRow + dchunk, dv1 = (uint32_t)(drow + 4) * kYRow + dchunk;
    const uint32_t mpad = (uint32_t)rmoff + (uint32_t)((rows + 3) / 4 * 4);   // staged mask bytes
    auto decode = [&](int u, int& i, int& j0) {
        i = u / nchunk;
        j0 = (u - i * nchunk) * kP3;
    };
    auto issue = [&](int u, int stage) {
        const bool valid = u < nunits;
        int i = 0, j0 = 0;
        if (valid) decode(u, i, j0);
        const int np = valid ? min(kP3, cols - j0) : 0;
        const uint32_t st = ring_base + (uint32_t)(stage * kRSt);
        const v4i_t rc = buffer_desc(C + result_off(nchunk, kCh, 0, i, j0), valid ? (uint32_t)kRC : 0u);
#pragma unroll
        for (int k = 0; k < 4; ++k) lds_load16(rc, cvo[k >> 1] + k * 1024, 0, st + w * 4096 + k * 1024);
        const v4i_t rz = buffer_desc(z + ((int64_t)i * cols + j0) * kCz, (uint32_t)np * kYRow);
        lds_load16(rz, dv0, 0, st + kRC + w * 2048);
        lds_load16(rz, dv1, 0, st + kRC + w * 2048 + 1024);
        const v4i_t rm = buffer_desc(tmask, valid ? mpad : 0u);
        const uint32_t mo = lane < 8 ? (uint32_t)(j0 + 4 * lane) : lane == 8 ? (uint32_t)(rmoff + (i & ~3)) : 0xfffffff0u;
        lds_load4(rm, mo, 0, st + kRC + kRZ + w * 256);
    };
    issue(first, 0);
    if (kStages == 3) issue(first + G, 1);

    bf16x8_t wo[8], wg[8];
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
        const size_t col = (size_t)ks * 16 + 8 * (lane >> 5);
        wo[ks] = *reinterpret_cast<const bf16x8_t*>(wepi + (size_t)(w * 32 + (lane & 31)) * 128 + col);
        wg[ks] = *reinterpret_cast<const bf16x8_t*>(wepi + (size_t)(128 + w * 32 + (lane & 31)) * 128 + col);
    }
    if (t < 128) {
        const int tp = (t >> 4) * 20 + (t & 15);
        prm[0][tp] = lnout_w[t];
        prm[1][tp] = lnout_b[t];
        prm[2][tp] = lnin_w[t];
        prm[3][tp] = lnin_b[t];
    }

    int stage = 0;
    for (int it = 0, u = first; u < nunits; ++it, u += G) {
        // Wait for this unit's loads.  Issued after them: two stages, the
        // stores of the previous unit; three stages, the next unit's loads
        // (7) and the stores of the units in between.
        if (kStages == 2) {
            if (it == 0) wait_vmcnt_pinned<0>();
            else wait_vmcnt_pinned<kS>();
        } else {
            if (it == 0) wait_vmcnt_pinned<7>();
            else if (it == 1) wait_vmcnt_pinned<7 + kS>();
            else wait_vmcnt_pinned<kS + 7 + kS>();
        }
        __syncthreads();
        // into the stage of the previous unit
        issue(u + (kStages - 1) * G, stage == 0 ? kStages - 1 : stage - 1);
        char* st = ring + stage * kRSt;
        stage = stage == kStages - 1 ? 0 : stage + 1;

        // LN_out over the 128 hidden channels of pair lp and LN_in over the
        // 128 pair channels, both from the stage; lane lq holds channels
        // 16 lq .. 16 lq + 15 of each.
        float v[16];
        {
            const char* crow = st + (16 * lq) * 128 + (lp & 3) * 4;
#pragma unroll
            for (int k = 0; k < 16; ++k)
                v[k] = *reinterpret_cast<const float*>(crow + k * 128 + (((lp >> 2) ^ ((k + lq) & 7)) << 4));
        }
        float zv[16];
        {
            const char* zr = st + kRC + lp * kYRow;
            const uint4 z0 = *reinterpret_cast<const uint4*>(zr + (((2 * lq) ^ (lp & 1)) << 4));
            const uint4 z1 = *reinterpret_cast<const uint4*>(zr + (((2 * lq + 1) ^ (lp & 1)) << 4));
            const uint32_t uu[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                zv[2 * k] = __uint_as_float(uu[k] << 16);
                zv[2 * k + 1] = __uint_as_float(uu[k] & 0xffff0000u);
            }
        }
        const uint8_t* ms = reinterpret_cast<const uint8_t*>(st + kRC + kRZ + w * 256);
        int ui, uj0;
        decode(u, ui, uj0);
        // Masked pairs (and tail pairs, whose staged mask is zero) get y = 0:
        // W_o y, and so the output, is then exactly 0 (no bias).
        const uint32_t keep = (ms[lp] & ms[32 + (ui & 3)]) ? 0xffffffffu : 0u;
        __syncthreads();   // every thread has read its C and z; the stage becomes y_hi, y_lo, x_hi

        {
            float s1 = 0.f;
#pragma unroll
            for (int k = 0; k < 16; ++k) s1 += v[k];
            s1 = sum_lanes8(s1);
            const float mu = s1 * (1.0f / kCh);
            float q2 = 0.f;
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                v[k] -= mu;
                q2 += v[k] * v[k];
            }
            q2 = sum_lanes8(q2);
            const float rs = rsqrtf(q2 * (1.0f / kCh) + eps);
            uint32_t yh[8], yl[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int c = 20 * lq + 2 * k;   // channel 16 lq + 2 k in prm
                const float y0 = v[2 * k] * rs * prm[0][c] + prm[1][c];
                const float y1 = v[2 * k + 1] * rs * prm[0][c + 1] + prm[1][c + 1];
                const uint32_t h = pack_bf16x2(y0, y1);
                yh[k] = h & keep;
                yl[k] = pack_bf16x2(y0 - __uint_as_float(h << 16), y1 - __uint_as_float(h & 0xffff0000u)) & keep;
            }
            *reinterpret_cast<uint4*>(st + yoff(lp, 2 * lq)) = make_uint4(yh[0], yh[1], yh[2], yh[3]);
            *reinterpret_cast<uint4*>(st + yoff(lp, 2 * lq + 1)) = make_uint4(yh[4], yh[5], yh[6], yh[7]);
            *reinterpret_cast<uint4*>(st + 8192 + yoff(lp, 2 * lq)) = make_uint4(yl[0], yl[1], yl[2], yl[3]);
            *reinterpret_cast<uint4*>(st + 8192 + yoff(lp, 2 * lq + 1)) = make_uint4(yl[4], yl[5], yl[6], yl[7]);
        }
        {
            float s1 = 0.f;
#pragma unroll
            for (int k = 0; k < 16; ++k) s1 += zv[k];
            s1 = sum_lanes8(s1);
            const float mu = s1 * (1.0f / kCz);
            float q2 = 0.f;
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                zv[k] -= mu;
                q2 += zv[k] * zv[k];
            }
            q2 = sum_lanes8(q2);
            const float rs = rsqrtf(q2 * (1.0f / kCz) + eps);
            uint32_t hx[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int c = 20 * lq + 2 * k;   // channel 16 lq + 2 k in prm
                hx[k] = pack_bf16x2(zv[2 * k] * rs * prm[2][c] + prm[3][c], zv[2 * k + 1] * rs * prm[2][c + 1] + prm[3][c + 1]);
            }
            *reinterpret_cast<uint4*>(st + kRC + yoff(lp, 2 * lq)) = make_uint4(hx[0], hx[1], hx[2], hx[3]);
            *reinterpret_cast<uint4*>(st + kRC + yoff(lp, 2 * lq + 1)) = make_uint4(hx[4], hx[5], hx[6], hx[7]);
        }
        __syncthreads();

        f32x16_t ay, ag;
#pragma unroll
        for (int r = 0; r < 16; ++r) ay[r] = ag[r] = 0.f;
        const int ap = lane & 31;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            const uint32_t o = yoff(ap, 2 * ks + (lane >> 5));
            const bf16x8_t yh = *reinterpret_cast<const bf16x8_t*>(st + o);
            const bf16x8_t yl = *reinterpret_cast<const bf16x8_t*>(st + 8192 + o);
            const bf16x8_t xh = *reinterpret_cast<const bf16x8_t*>(st + kRC + o);
            ay = __builtin_amdgcn_mfma_f32_32x32x16_bf16(yh, wo[ks], ay, 0, 0, 0);
            ag = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xh, wg[ks], ag, 0, 0, 0);
            ay = __builtin_amdgcn_mfma_f32_32x32x16_bf16(yl, wo[ks], ay, 0, 0, 0);
        }

        // Lane holds output channel 32 w + (lane & 31); register r holds pair
        // 8 (r / 4) + 4 (lane / 32) + r % 4 (tail pairs come out as zeros and
        // are not stored).
        const int d = w * 32 + (lane & 31);
        const int np = min(kP3, cols - uj0);
        if constexpr (kDirect) {
            // bytes past the row's last pair fall outside the descriptor
            const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + ((int64_t)ui * cols + uj0) * kCz,
                                                        (uint32_t)(np * kCz * 4));
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int p = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(sigmoidf_(ag[r]) * ay[r]), ro,
                                                      (p * kCz + d) * 4, 0, 0);
            }
            continue;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int p = 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            os[p * kOsRow + d] = sigmoidf_(ag[r]) * ay[r];
        }
        __syncthreads();

        // bf16: the unit's [32 pairs][128] block is contiguous in out: store k
        // of the work-group covers its bytes [4096 k, 4096 k + 4096), 16 per
        // thread; bytes past the row's last pair fall outside the descriptor.
        const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + ((int64_t)ui * cols + uj0) * kCz,
                                                    (uint32_t)(np * kCz * (int)sizeof(TO)));
#pragma unroll
        for (int k = 0; k < kStores; ++k) {
            const uint32_t off = (uint32_t)(k * 4096 + t * 16);
            const int p = off / 256, d8 = (off % 256) / 2;
            const float4 f0 = *reinterpret_cast<const float4*>(&os[p * kOsRow + d8]);
            const float4 f1 = *reinterpret_cast<const float4*>(&os[p * kOsRow + d8 + 4]);
            const uint4 pk = make_uint4(pack_bf16x2(f0.x, f0.y), pack_bf16x2(f0.z, f0.w), pack_bf16x2(f1.x, f1.y),
                                        pack_bf16x2(f1.z, f1.w));
            __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i_t, pk), ro, off, 0, 0);
        }
    }
    wait_vmcnt_pinned<0>();   // the ring load past the last unit lands before the work-group ends
}

template <typename T, typename TO>
hipError_t launch_valu(const DeviceWeights& w, const EpilogueArgs& a, hipStream_t s) {
    const int64_t nchunk = (a.cols + kPairs - 1) / kPairs;
    hipLaunchKernelGGL((k3_epilogue_valu<T, TO>), dim3((unsigned)(a.rows * nchunk)), dim3(256), 0, s, a,
                       nchunk, w.wo_t, w.wg_t, w.ln_in_w, w.ln_in_b, w.ln_out_w, w.ln_out_b, w.eps);
    return hipGetLastError();
}

template <typename TO>
hipError_t launch_mfma(const DeviceWeights& w, const EpilogueArgs& a, hipStream_t s) {
    const int nchunk = (int)((a.cols + kP3 - 1) / kP3);
    const int64_t nunits = a.rows * nchunk;
    const int64_t cap = 2 * (int64_t)w.cus;
    const unsigned g = (unsigned)(nunits < cap ? nunits : cap);
    const bool vec = (a.ldc % 4) == 0 && (a.sc % 4) == 0 && (reinterpret_cast<uintptr_t>(a.C) & 15u) == 0;
    if (a.cblocked) {   // C in the pair-blocked layout: the full update, or a tile's packed accumulator
        const int rmoff = (int)((a.cols + 31) / 32 * 32);
        hipError_t e = launch_stage_tile_mask(a.mask, a.row0, a.rows, a.col0, a.cols, w.kmask_pad, s);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((k3_epilogue_ring<TO>), dim3(g), dim3(256), 0, s, a.C, (const bf16_t*)a.z, w.kmask_pad,
                           (int)a.rows, (int)a.cols, rmoff, (int)nunits, (TO*)a.out, w.epi_bf, w.ln_in_w, w.ln_in_b,
                           w.ln_out_w, w.ln_out_b, w.eps);
    } else if (vec)
        hipLaunchKernelGGL((k3_epilogue_mfma<TO, true, false>), dim3(g), dim3(256), 0, s, a, nchunk, nunits, w.epi_bf,
                           w.ln_in_w, w.ln_in_b, w.ln_out_w, w.ln_out_b, w.eps);
    else
        hipLaunchKernelGGL((k3_epilogue_mfma<TO, false, false>), dim3(g), dim3(256), 0, s, a, nchunk, nunits, w.epi_bf,
                           w.ln_in_w, w.ln_in_b, w.ln_out_w, w.ln_out_b, w.eps);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_epilogue(int dtype, int out_dtype, const DeviceWeights& w, const EpilogueArgs& a,
                           hipStream_t s) {
    if (dtype == 0)
        return out_dtype == 0 ? launch_valu<float, float>(w, a, s) : launch_valu<float, bf16_t>(w, a, s);
    return out_dtype == 0 ? launch_mfma<float>(w, a, s) : launch_mfma<bf16_t>(w, a, s);
}

}  // namespace trimul
