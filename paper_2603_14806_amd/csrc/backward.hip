// Backward of the per-channel contraction (training; the paper gives every
// distributed module an explicit backward that runs the same schedule as its
// forward, Section 3.1).  With the channel-major operands of the forward,
// C[c] = A[c] B[c]^T, the gradients are two more products of the same size:
//
//     dA[c] = dC[c] B[c]        dB[c] = dC[c]^T A[c]
//
// and both are again "NT" products once the right operands are transposed:
// dA = NT(dC, B^T), dB = NT(dC^T, A^T).  This file holds the two layout
// kernels that prepare those operands in the blocked panel layout; the
// products run on the contraction kernels.
#include "common.h"
#include "kernels.h"

namespace trimul {
namespace {

// dC in the pair-blocked result layout (fp32) -> the panel layout, element
// (c, i, j) -> X_c[i][k = j], converted to T.  One unit = one row i and one
// 32-column block: 128 channels x 32 floats, contiguous in both layouts per
// channel.  Thread t moves channel t / 2, columns 16 (t % 2) .. + 15.
// Columns past N carry whatever the result layout holds there into the k
// padding of the panel, which the contraction never uses.
template <typename T>
__global__ __launch_bounds__(256) void k_result_to_panel(const float* __restrict__ R, T* __restrict__ P, int N,
                                                        int64_t units) {
    const int t = threadIdx.x, ch = t >> 1, h = t & 1;
    const int J = (N + kResJ - 1) / kResJ;
    const PanelGeom pg = panel_geom(N, N);
    for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
        const int64_t i = u / J, jb = u - (u / J) * J;
        const float4* src = reinterpret_cast<const float4*>(R + result_off(J, kCh, ch, i, jb * kResJ) + 16 * h);
        float4 v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = src[q];
        T* dst = P + panel_off(pg, ch, i, jb * kResJ + 16 * h);
        if constexpr (sizeof(T) == 2) {
            uint4 o[2];
            o[0] = make_uint4(pack_bf16x2(v[0].x, v[0].y), pack_bf16x2(v[0].z, v[0].w),
                              pack_bf16x2(v[1].x, v[1].y), pack_bf16x2(v[1].z, v[1].w));
            o[1] = make_uint4(pack_bf16x2(v[2].x, v[2].y), pack_bf16x2(v[2].z, v[2].w),
                              pack_bf16x2(v[3].x, v[3].y), pack_bf16x2(v[3].z, v[3].w));
            reinterpret_cast<uint4*>(dst)[0] = o[0];
            reinterpret_cast<uint4*>(dst)[1] = o[1];
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) reinterpret_cast<float4*>(dst)[q] = v[q];
        }
    }
}

// Per-channel transpose in the panel layout: Y_c[k][i] = X_c[i][k].  One wave
// moves one 32 x 32 block (rows 32 ib.., columns 32 kb..) through LDS: lane l
// reads 16 consecutive elements of row l / 2 (half l % 2) and writes 16
// consecutive elements of output row l / 2.  Blocks cover [0, 32 S)^2 with
// S = ceil(N / 32), which lies inside the panel allocation; padding elements
// move along with the rest.
template <typename T>
__global__ __launch_bounds__(256) void k_panel_transpose(const T* __restrict__ X, T* __restrict__ Y, int N,
                                                        int64_t blocks) {
    constexpr int kPad = 34;   // row stride (elements) of the wave's tile
    __shared__ T tile[4][32 * kPad];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int S = (N + 31) / 32;
    const PanelGeom pg = panel_geom(N, N);
    const int rr = lane >> 1, hh = lane & 1;
    T* tl = tile[w];
    const int64_t waves = (int64_t)gridDim.x * 4;
    for (int64_t b = (int64_t)blockIdx.x * 4 + w; b < blocks; b += waves) {
        const int64_t ch = b / ((int64_t)S * S);
        const int64_t rem = b - ch * S * S;
        const int ib = (int)(rem / S), kb = (int)(rem - (int64_t)(rem / S) * S);
        const T* src = X + panel_off(pg, ch, 32 * ib + rr, 32 * kb + 16 * hh);   // 16 elements, 32 B aligned
        T* dst = Y + panel_off(pg, ch, 32 * kb + rr, 32 * ib + 16 * hh);
        T* trow = tl + rr * kPad + 16 * hh;
        if constexpr (sizeof(T) == 2) {
            const uint4 a0 = reinterpret_cast<const uint4*>(src)[0], a1 = reinterpret_cast<const uint4*>(src)[1];
            const uint32_t w8[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
#pragma unroll
            for (int q = 0; q < 8; ++q) reinterpret_cast<uint32_t*>(trow)[q] = w8[q];
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 f = reinterpret_cast<const float4*>(src)[q];
                reinterpret_cast<float*>(trow)[4 * q] = f.x;
                reinterpret_cast<float*>(trow)[4 * q + 1] = f.y;
                reinterpret_cast<float*>(trow)[4 * q + 2] = f.z;
                reinterpret_cast<float*>(trow)[4 * q + 3] = f.w;
            }
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        T v[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) v[q] = tl[(16 * hh + q) * kPad + rr];
        if constexpr (sizeof(T) == 2) {
            uint32_t w8[8];
#pragma unroll
            for (int q = 0; q < 8; ++q)
                w8[q] = (uint32_t)__builtin_bit_cast(uint16_t, v[2 * q]) |
                        ((uint32_t)__builtin_bit_cast(uint16_t, v[2 * q + 1]) << 16);
            reinterpret_cast<uint4*>(dst)[0] = make_uint4(w8[0], w8[1], w8[2], w8[3]);
            reinterpret_cast<uint4*>(dst)[1] = make_uint4(w8[4], w8[5], w8[6], w8[7]);
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                reinterpret_cast<float4*>(dst)[q] = make_float4(__builtin_bit_cast(float, v[4 * q]),
                                                                __builtin_bit_cast(float, v[4 * q + 1]),
                                                                __builtin_bit_cast(float, v[4 * q + 2]),
                                                                __builtin_bit_cast(float, v[4 * q + 3]));
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    }
}

// ---------------------------------------------------------------- layer backward
//
// Work unit = 32 pairs (one row r, columns k = 32 kb .. 32 kb + 31), the
// unit of the result layout.  Per-pair intermediates that feed the weight
// gradients are written as "unit blocks": for unit u = r * J + kb, a bf16
// block [128 channels][32 slots] at u * 4096 elements; slots of pairs past N
// hold zeros.  Each weight gradient is then a sum over units of
// U_block * V_block^T (k_wgrad).  The per-pair stages here are fp32 VALU
// kernels (4 x 4 register tiles per thread over an LDS copy of the unit).
constexpr int kQ = 32;              // pairs per unit
constexpr int kRow = 129;           // LDS row stride (floats) of [pair][channel] tiles
constexpr int kCol = 33;            // LDS row stride (floats) of [channel][pair] tiles
constexpr int kCol4 = 36;           // the same, 16-byte aligned rows (read as float4)

__device__ __forceinline__ float bfr(float v) { return bf2f(f2bf(v)); }

// 16 consecutive floats -> 16 bf16 (32 bytes) at dst.
__device__ __forceinline__ void st16bf(bf16_t* dst, const float (&v)[16]) {
    uint4 o0 = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
    uint4 o1 = make_uint4(pack_bf16x2(v[8], v[9]), pack_bf16x2(v[10], v[11]), pack_bf16x2(v[12], v[13]),
                          pack_bf16x2(v[14], v[15]));
    reinterpret_cast<uint4*>(dst)[0] = o0;
    reinterpret_cast<uint4*>(dst)[1] = o1;
}

template <typename T> __device__ __forceinline__ float ldv(const T* p);
template <> __device__ __forceinline__ float ldv<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ldv<bf16_t>(const bf16_t* p) { return bf2f(*p); }

// Epilogue backward.  For the unit's pairs (r, k): recompute x = LN_in(z),
// y = LN_out(C), u = W_o y, g = sigmoid(W_g x); then
//   du = dout m g,  dgg = dout m u g (1 - g),  dy = du W_o,  dx_g = dgg W_g,
//   dC = LN_out backward of dy.
// Writes dC into the panel (rows r, k), dx_g [pair][c_z] fp32, unit blocks
// du, y, dgg, x, and per-work-group partial sums of dgamma_out, dbeta_out.
template <typename T, typename TO>
__global__ __launch_bounds__(256) void k_epilogue_backward(
    const float* __restrict__ C, const T* __restrict__ z, const uint8_t* __restrict__ mask, const TO* __restrict__ dout,
    int N, int64_t units, const float* __restrict__ wo_t, const float* __restrict__ wg_t, const float* __restrict__ wo,
    const float* __restrict__ wg, const float* __restrict__ lniw, const float* __restrict__ lnib,
    const float* __restrict__ lnow, const float* __restrict__ lnob, float eps, T* __restrict__ dCp,
    float* __restrict__ dxg, bf16_t* __restrict__ b_du, bf16_t* __restrict__ b_y, bf16_t* __restrict__ b_dgg,
    bf16_t* __restrict__ b_x, float* __restrict__ partial) {
    __shared__ float cs[kCh * kCol];      // C [c][q]
    __shared__ float xs[kQ * kRow];       // z, then x [q][d]
    __shared__ float ds[kQ * kRow];       // dout [q][d], then dy [q][c]
    __shared__ float ys[kQ * kRow];       // y [q][c]
    __shared__ float yh[kQ * kRow];       // normalised C [q][c]
    __shared__ float us[kQ * kRow];       // du [q][d]
    __shared__ float gs[kQ * kRow];       // dgg [q][d]
    __shared__ float st[3][kQ];           // rstd, mean(dyhat), mean(dyhat * yhat)
    __shared__ float mq[kQ];              // pair mask
    const int t = threadIdx.x;
    const int J = (N + kQ - 1) / kQ;
    const PanelGeom pg = panel_geom(N, N);
    const int lp = t >> 3, lq = t & 7;                 // LayerNorms: pair lp, 8 lanes per pair
    const int tg = t & 31, tq = t >> 5;                // matvecs: outputs 4 tg .. + 3, pairs 4 tq .. + 3
    const int pc = t >> 1, ph = t & 1;                 // channel-major passes: channel pc, pairs 16 ph .. + 15
    float acc_g = 0.f, acc_b = 0.f;                    // dgamma_out, dbeta_out of channel pc, pairs of half ph

    for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
        const int r = (int)(u / J), kb = (int)(u - (int64_t)r * J);
        const int k0 = kb * kQ;
        // (1) loads
        {
            // C's columns past N hold unspecified values: read them as zero
            const float4* cb = reinterpret_cast<const float4*>(C + u * (kCh * kQ));
            const int nq = N - k0;
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) {
                const int e = 4 * (t + 256 * s2), ch = e >> 5, q = e & 31;
                const float4 v = cb[t + 256 * s2];
                cs[ch * kCol + q] = q < nq ? v.x : 0.f;
                cs[ch * kCol + q + 1] = q + 1 < nq ? v.y : 0.f;
                cs[ch * kCol + q + 2] = q + 2 < nq ? v.z : 0.f;
                cs[ch * kCol + q + 3] = q + 3 < nq ? v.w : 0.f;
            }
            const bool valid = k0 + lp < N;
            const int64_t pr = (int64_t)r * N + k0 + lp;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int d = 16 * lq + i;
                xs[lp * kRow + d] = valid ? ldv<T>(z + pr * kCz + d) : 0.f;
                ds[lp * kRow + d] = valid ? ldv<TO>(dout + pr * kCz + d) : 0.f;
            }
            if (t < kQ) {
                const int k = k0 + t;
                mq[t] = (k < N && (!mask || (mask[r] != 0 && mask[k] != 0))) ? 1.f : 0.f;
            }
        }
        __syncthreads();
        // (2) LN_out over c for pair lp (lane lq: c = lq + 8 i), LN_in over d (16 lq + i)
        {
            float v[16], s1 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) { v[i] = cs[(lq + 8 * i) * kCol + lp]; s1 += v[i]; }
            s1 = sum_lanes8(s1);
            const float mu = s1 * (1.f / kCh);
            float q2 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) { v[i] -= mu; q2 += v[i] * v[i]; }
            q2 = sum_lanes8(q2);
            const float rs = rsqrtf(q2 * (1.f / kCh) + eps);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int c = lq + 8 * i;
                yh[lp * kRow + c] = v[i] * rs;
                ys[lp * kRow + c] = v[i] * rs * lnow[c] + lnob[c];
            }
            if (lq == 0) st[0][lp] = rs;
            float w[16];
            s1 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) { w[i] = xs[lp * kRow + 16 * lq + i]; s1 += w[i]; }
            s1 = sum_lanes8(s1);
            const float mz = s1 * (1.f / kCz);
            q2 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) { w[i] -= mz; q2 += w[i] * w[i]; }
            q2 = sum_lanes8(q2);
            const float rz = rsqrtf(q2 * (1.f / kCz) + eps);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int d = 16 * lq + i;
                xs[lp * kRow + d] = w[i] * rz * lniw[d] + lnib[d];
            }
        }
        __syncthreads();
        // (3) u = W_o y, gg = W_g x; du, dgg
        {
            float au[4][4] = {}, ag[4][4] = {};
            for (int c = 0; c < kCh; ++c) {
                const float4 wu = *reinterpret_cast<const float4*>(wo_t + c * kCz + 4 * tg);
                const float4 wv = *reinterpret_cast<const float4*>(wg_t + c * kCz + 4 * tg);
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    const float yv = ys[(4 * tq + a) * kRow + c], xv = xs[(4 * tq + a) * kRow + c];
                    au[a][0] += yv * wu.x; au[a][1] += yv * wu.y; au[a][2] += yv * wu.z; au[a][3] += yv * wu.w;
                    ag[a][0] += xv * wv.x; ag[a][1] += xv * wv.y; ag[a][2] += xv * wv.z; ag[a][3] += xv * wv.w;
                }
            }
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const int q = 4 * tq + a;
                const float m = mq[q];
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const int d = 4 * tg + b;
                    const float g = 1.f / (1.f + __expf(-ag[a][b]));
                    const float o = ds[q * kRow + d] * m;
                    us[q * kRow + d] = o * g;
                    gs[q * kRow + d] = o * au[a][b] * g * (1.f - g);
                }
            }
        }
        __syncthreads();
        // (4) dy = du W_o (into ds), dx_g = dgg W_g (to HBM)
        {
            float ay[4][4] = {}, ax[4][4] = {};
            for (int d = 0; d < kCz; ++d) {
                const float4 wu = *reinterpret_cast<const float4*>(wo + d * kCh + 4 * tg);
                const float4 wv = *reinterpret_cast<const float4*>(wg + d * kCz + 4 * tg);
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    const float uv = us[(4 * tq + a) * kRow + d], gv = gs[(4 * tq + a) * kRow + d];
                    ay[a][0] += uv * wu.x; ay[a][1] += uv * wu.y; ay[a][2] += uv * wu.z; ay[a][3] += uv * wu.w;
                    ax[a][0] += gv * wv.x; ax[a][1] += gv * wv.y; ax[a][2] += gv * wv.z; ax[a][3] += gv * wv.w;
                }
            }
#pragma unroll
            for (int a = 0; a < 4; ++a) {
                const int q = 4 * tq + a;
#pragma unroll
                for (int b = 0; b < 4; ++b) ds[q * kRow + 4 * tg + b] = ay[a][b];
                if (k0 + q < N)
                    *reinterpret_cast<float4*>(dxg + ((int64_t)r * N + k0 + q) * kCz + 4 * tg) =
                        make_float4(ax[a][0], ax[a][1], ax[a][2], ax[a][3]);
            }
        }
        __syncthreads();
        // (5) LN_out backward statistics of pair lp
        {
            float s1 = 0.f, s2 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int c = lq + 8 * i;
                const float dh = ds[lp * kRow + c] * lnow[c];
                s1 += dh;
                s2 += dh * yh[lp * kRow + c];
            }
            s1 = sum_lanes8(s1);
            s2 = sum_lanes8(s2);
            if (lq == 0) { st[1][lp] = s1 * (1.f / kCh); st[2][lp] = s2 * (1.f / kCh); }
        }
        __syncthreads();
        // (6) channel-major outputs: dC into the panel, unit blocks, dgamma / dbeta
        {
            float dc[16], v0[16], v1[16], v2[16], v3[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int q = 16 * ph + i;
                const bool ok = k0 + q < N;
                const float dy = ds[q * kRow + pc], yv = yh[q * kRow + pc];
                dc[i] = st[0][q] * (dy * lnow[pc] - st[1][q] - yv * st[2][q]);
                acc_g += dy * yv;
                acc_b += dy;
                v0[i] = us[q * kRow + pc];
                v1[i] = ok ? ys[q * kRow + pc] : 0.f;
                v2[i] = gs[q * kRow + pc];
                v3[i] = ok ? xs[q * kRow + pc] : 0.f;
            }
            T* dst = dCp + panel_off(pg, pc, r, k0 + 16 * ph);
            if constexpr (sizeof(T) == 2) {
                st16bf(dst, dc);
            } else {
#pragma unroll
                for (int i = 0; i < 16; ++i) dst[i] = dc[i];
            }
            const int64_t bo = u * (kCh * kQ) + pc * kQ + 16 * ph;
            st16bf(b_du + bo, v0);
            st16bf(b_y + bo, v1);
            st16bf(b_dgg + bo, v2);
            st16bf(b_x + bo, v3);
        }
        __syncthreads();
    }
    partial[((int64_t)blockIdx.x * 4 + 2 * ph + 0) * kCh + pc] = acc_g;
    partial[((int64_t)blockIdx.x * 4 + 2 * ph + 1) * kCh + pc] = acc_b;
}

// Projection backward.  Unit (r, kb) of dA / dB; its pairs are P(q) = (r, k)
// (outgoing) or (k, r) (incoming).  Recompute x = LN_in(z) and the four
// projections; then dpa = da m s_a, dga = da m p_a s_a (1 - s_a) (same for b),
// dx = dx_g + W_a^T dpa + W_ga^T dga + W_b^T dpb + W_gb^T dgb, and
// dz = LN_in backward of dx.  Writes dz, unit blocks dpa, dga, dpb, dgb, x,
// and per-work-group partial sums of dgamma_in, dbeta_in.
template <typename T, bool INCOMING>
__global__ __launch_bounds__(256) void k_projection_backward(
    const T* __restrict__ z, const uint8_t* __restrict__ mask, int N, int64_t units, const float* __restrict__ dA,
    const float* __restrict__ dB, const float* __restrict__ dxg, const float4* __restrict__ proj4,
    const float4* __restrict__ projb, const float* __restrict__ lniw, const float* __restrict__ lnib, float eps,
    T* __restrict__ dz, bf16_t* __restrict__ b_dpa, bf16_t* __restrict__ b_dga, bf16_t* __restrict__ b_dpb,
    bf16_t* __restrict__ b_dgb, bf16_t* __restrict__ b_x, float* __restrict__ partial) {
    __shared__ float zs[kQ * kRow];       // z [q][d]
    __shared__ float xs[kQ * kRow];       // x [q][d]
    __shared__ float gx[kQ * kRow];       // dx_g, then dx [q][d]
    __shared__ float das[kCh * kCol];     // da [c][q]
    __shared__ float dbs[kCh * kCol];     // db [c][q]
    __shared__ __align__(16) float d4[4][kCh * kCol4];  // dpa, dga, dpb, dgb [c][q]
    __shared__ float st[4][kQ];           // mean, rstd, mean(dxhat), mean(dxhat * xhat)
    __shared__ float mq[kQ];
    const int t = threadIdx.x;
    const int J = (N + kQ - 1) / kQ;
    const int lp = t >> 3, lq = t & 7;
    const int tg = t & 31, tq = t >> 5;
    const int pc = t & 127, ph = t >> 7;               // projections: channel pc, pairs 16 ph .. + 15
    const int bc = t >> 1, bh = t & 1;                 // x block: channel bc, pairs 16 bh .. + 15
    float acc_g[16], acc_b[16];                        // dgamma_in, dbeta_in for d = 16 lq + i
#pragma unroll
    for (int i = 0; i < 16; ++i) acc_g[i] = acc_b[i] = 0.f;
    auto pair_of = [&](int r, int k) -> int64_t { return INCOMING ? (int64_t)k * N + r : (int64_t)r * N + k; };

    for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
        const int r = (int)(u / J), kb = (int)(u - (int64_t)r * J);
        const int k0 = kb * kQ;
        {
            const float4* ab = reinterpret_cast<const float4*>(dA + u * (kCh * kQ));
            const float4* bb = reinterpret_cast<const float4*>(dB + u * (kCh * kQ));
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) {
                const int e = 4 * (t + 256 * s2), ch = e >> 5, q = e & 31;
                const float4 a = ab[t + 256 * s2], b = bb[t + 256 * s2];
                das[ch * kCol + q] = a.x; das[ch * kCol + q + 1] = a.y; das[ch * kCol + q + 2] = a.z; das[ch * kCol + q + 3] = a.w;
                dbs[ch * kCol + q] = b.x; dbs[ch * kCol + q + 1] = b.y; dbs[ch * kCol + q + 2] = b.z; dbs[ch * kCol + q + 3] = b.w;
            }
            const bool valid = k0 + lp < N;
            const int64_t pr = valid ? pair_of(r, k0 + lp) : 0;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int d = 16 * lq + i;
                zs[lp * kRow + d] = valid ? ldv<T>(z + pr * kCz + d) : 0.f;
                gx[lp * kRow + d] = valid ? dxg[pr * kCz + d] : 0.f;
            }
            if (t < kQ) {
                const int k = k0 + t;
                mq[t] = (k < N && (!mask || (mask[r] != 0 && mask[k] != 0))) ? 1.f : 0.f;
            }
        }
        __syncthreads();
        {   // LN_in of pair lp
            float w[16], s1 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) { w[i] = zs[lp * kRow + 16 * lq + i]; s1 += w[i]; }
            s1 = sum_lanes8(s1);
            const float mz = s1 * (1.f / kCz);
            float q2 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) { w[i] -= mz; q2 += w[i] * w[i]; }
            q2 = sum_lanes8(q2);
            const float rz = rsqrtf(q2 * (1.f / kCz) + eps);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int d = 16 * lq + i;
                xs[lp * kRow + d] = w[i] * rz * lniw[d] + lnib[d];
            }
            if (lq == 0) { st[0][lp] = mz; st[1][lp] = rz; }
        }
        __syncthreads();
        {   // projections of channel pc for 16 pairs, then the four gradients
            float acc[16][4];
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[i][0] = acc[i][1] = acc[i][2] = acc[i][3] = 0.f;
            for (int d = 0; d < kCz; ++d) {
                const float4 w = proj4[d * kCh + pc];
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const float xv = xs[(16 * ph + i) * kRow + d];
                    acc[i][0] += w.x * xv; acc[i][1] += w.y * xv; acc[i][2] += w.z * xv; acc[i][3] += w.w * xv;
                }
            }
            float o0[16], o1[16], o2[16], o3[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int q = 16 * ph + i;
                const bool m = mq[q] != 0.f;
                const float sa = 1.f / (1.f + __expf(-acc[i][1])), sb = 1.f / (1.f + __expf(-acc[i][3]));
                const float da = das[pc * kCol + q], db = dbs[pc * kCol + q];
                o0[i] = m ? da * sa : 0.f;
                o1[i] = m ? da * acc[i][0] * sa * (1.f - sa) : 0.f;
                o2[i] = m ? db * sb : 0.f;
                o3[i] = m ? db * acc[i][2] * sb * (1.f - sb) : 0.f;
                d4[0][pc * kCol4 + q] = o0[i];
                d4[1][pc * kCol4 + q] = o1[i];
                d4[2][pc * kCol4 + q] = o2[i];
                d4[3][pc * kCol4 + q] = o3[i];
            }
            const int64_t bo = u * (kCh * kQ) + pc * kQ + 16 * ph;
            st16bf(b_dpa + bo, o0);
            st16bf(b_dga + bo, o1);
            st16bf(b_dpb + bo, o2);
            st16bf(b_dgb + bo, o3);
        }
        __syncthreads();
        {   // dx = dx_g + sum over the four maps of W^T (gradient)
            float ax[4][4];
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b) ax[a][b] = gx[(4 * tq + a) * kRow + 4 * tg + b];
            for (int c = 0; c < kCh; ++c) {
                float4 w[4];
#pragma unroll
                for (int b = 0; b < 4; ++b) w[b] = projb[c * kCz + 4 * tg + b];
                const float4 g0 = *reinterpret_cast<const float4*>(&d4[0][c * kCol4 + 4 * tq]);
                const float4 g1 = *reinterpret_cast<const float4*>(&d4[1][c * kCol4 + 4 * tq]);
                const float4 g2 = *reinterpret_cast<const float4*>(&d4[2][c * kCol4 + 4 * tq]);
                const float4 g3 = *reinterpret_cast<const float4*>(&d4[3][c * kCol4 + 4 * tq]);
                const float ga[4][4] = {{g0.x, g1.x, g2.x, g3.x}, {g0.y, g1.y, g2.y, g3.y},
                                        {g0.z, g1.z, g2.z, g3.z}, {g0.w, g1.w, g2.w, g3.w}};
#pragma unroll
                for (int a = 0; a < 4; ++a)
#pragma unroll
                    for (int b = 0; b < 4; ++b)
                        ax[a][b] += ga[a][0] * w[b].x + ga[a][1] * w[b].y + ga[a][2] * w[b].z + ga[a][3] * w[b].w;
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b) gx[(4 * tq + a) * kRow + 4 * tg + b] = ax[a][b];
        }
        __syncthreads();
        {   // LN_in backward of pair lp, dz, dgamma_in / dbeta_in
            const float mz = st[0][lp], rz = st[1][lp];
            float dh[16], xh[16], s1 = 0.f, s2 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int d = 16 * lq + i;
                const float dx = gx[lp * kRow + d];
                xh[i] = (zs[lp * kRow + d] - mz) * rz;
                dh[i] = dx * lniw[d];
                s1 += dh[i];
                s2 += dh[i] * xh[i];
                acc_g[i] += dx * xh[i];
                acc_b[i] += dx;
            }
            s1 = sum_lanes8(s1) * (1.f / kCz);
            s2 = sum_lanes8(s2) * (1.f / kCz);
            if (k0 + lp < N) {
                T* dst = dz + pair_of(r, k0 + lp) * kCz + 16 * lq;
                float o[16];
#pragma unroll
                for (int i = 0; i < 16; ++i) o[i] = rz * (dh[i] - s1 - xh[i] * s2);
                if constexpr (sizeof(T) == 2) {
                    st16bf(dst, o);
                } else {
#pragma unroll
                    for (int i = 0; i < 16; ++i) dst[i] = o[i];
                }
            }
            float v[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int q = 16 * bh + i;
                v[i] = (k0 + q < N) ? xs[q * kRow + bc] : 0.f;
            }
            st16bf(b_x + u * (kCh * kQ) + bc * kQ + 16 * bh, v);
        }
        __syncthreads();
    }
    // reduce the per-thread LayerNorm parameter sums over the 32 pairs lanes
    // (threads with the same lq) through LDS, then one partial per work-group
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        xs[lp * kRow + 16 * lq + i] = acc_g[i];
        zs[lp * kRow + 16 * lq + i] = acc_b[i];
    }
    __syncthreads();
    if (t < kCz) {
        float sg = 0.f, sb = 0.f;
        for (int q = 0; q < kQ; ++q) { sg += xs[q * kRow + t]; sb += zs[q * kRow + t]; }
        partial[((int64_t)blockIdx.x * 2 + 0) * kCz + t] = sg;
        partial[((int64_t)blockIdx.x * 2 + 1) * kCz + t] = sb;
    }
}

// Weight-gradient sum: W[m][n] = sum over units of U_blk[m][.] . V_blk[n][.]
// (both [128][32] bf16 unit blocks, the dot product over the 32 slots), on
// matrix cores: wave w owns rows 32 w .. 32 w + 31 and all 128 columns
// (4 blocks of v_mfma_f32_32x32x16_bf16, two k-steps per unit).  Each
// work-group writes one 128 x 128 fp32 partial.
__global__ __launch_bounds__(256) void k_wgrad(const bf16_t* __restrict__ U, const bf16_t* __restrict__ V,
                                                int64_t units, float* __restrict__ partial) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int rl = lane & 31, hi = lane >> 5;
    f32x16_t acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[j][r] = 0.f;
    for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
        const bf16_t* ub = U + u * (kCh * kQ);
        const bf16_t* vb = V + u * (kCh * kQ);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const bf16x8_t a = *reinterpret_cast<const bf16x8_t*>(ub + (32 * w + rl) * kQ + 16 * ks + 8 * hi);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bf16x8_t b = *reinterpret_cast<const bf16x8_t*>(vb + (32 * j + rl) * kQ + 16 * ks + 8 * hi);
                acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
            }
        }
    }
    // lane holds column 32 j + rl; register r holds row 32 w + 8 (r / 4) + 4 hi + r % 4
    float* pw = partial + (int64_t)blockIdx.x * (kCh * kCh);
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) pw[(32 * w + 8 * (r >> 2) + 4 * hi + (r & 3)) * kCh + 32 * j + rl] = acc[j][r];
}

// out[i] = sum over g < parts of in[g * stride + i], in that order.
__global__ __launch_bounds__(256) void k_sum_parts(const float* __restrict__ in, int parts, int64_t stride, int n,
                                                    float* __restrict__ out) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    float s = 0.f;
    for (int g = 0; g < parts; ++g) s += in[(int64_t)g * stride + i];
    out[i] = s;
}

}  // namespace

hipError_t launch_result_to_panel(int dtype, const float* R, void* P, int64_t N, int cus, hipStream_t s) {
    const int64_t units = N * ((N + kResJ - 1) / kResJ);
    const unsigned g = (unsigned)(units < 8 * (int64_t)cus ? units : 8 * (int64_t)cus);
    if (dtype == 0)
        hipLaunchKernelGGL(k_result_to_panel<float>, dim3(g), dim3(256), 0, s, R, (float*)P, (int)N, units);
    else
        hipLaunchKernelGGL(k_result_to_panel<bf16_t>, dim3(g), dim3(256), 0, s, R, (bf16_t*)P, (int)N, units);
    return hipGetLastError();
}

hipError_t launch_panel_transpose(int dtype, const void* X, void* Y, int64_t N, int cus, hipStream_t s) {
    const int64_t S = (N + 31) / 32;
    const int64_t blocks = (int64_t)kCh * S * S;
    const int64_t wgs = (blocks + 3) / 4;
    const unsigned g = (unsigned)(wgs < 8 * (int64_t)cus ? wgs : 8 * (int64_t)cus);
    if (dtype == 0)
        hipLaunchKernelGGL(k_panel_transpose<float>, dim3(g), dim3(256), 0, s, (const float*)X, (float*)Y, (int)N,
                           blocks);
    else
        hipLaunchKernelGGL(k_panel_transpose<bf16_t>, dim3(g), dim3(256), 0, s, (const bf16_t*)X, (bf16_t*)Y,
                           (int)N, blocks);
    return hipGetLastError();
}

}  // namespace trimul

namespace trimul {

int backward_grid(int64_t units, int cus) { return (int)(units < 2 * (int64_t)cus ? units : 2 * (int64_t)cus); }

hipError_t launch_epilogue_backward(int out_dtype, const DeviceWeights& w, const float* C, const void* z,
                                    const uint8_t* mask, const void* dout, int64_t N, void* dCp, float* dxg,
                                    const BackwardBlocks& bb, float* partial, int grid, hipStream_t s) {
    const int64_t units = N * ((N + 31) / 32);
    if (out_dtype == 0)
        hipLaunchKernelGGL((k_epilogue_backward<bf16_t, float>), dim3(grid), dim3(256), 0, s, C, (const bf16_t*)z, mask,
                           (const float*)dout, (int)N, units, w.wo_t, w.wg_t, w.wo, w.wg, w.ln_in_w, w.ln_in_b,
                           w.ln_out_w, w.ln_out_b, w.eps, (bf16_t*)dCp, dxg, bb.du, bb.y, bb.dgg, bb.xe, partial);
    else
        hipLaunchKernelGGL((k_epilogue_backward<bf16_t, bf16_t>), dim3(grid), dim3(256), 0, s, C, (const bf16_t*)z,
                           mask, (const bf16_t*)dout, (int)N, units, w.wo_t, w.wg_t, w.wo, w.wg, w.ln_in_w, w.ln_in_b,
                           w.ln_out_w, w.ln_out_b, w.eps, (bf16_t*)dCp, dxg, bb.du, bb.y, bb.dgg, bb.xe, partial);
    return hipGetLastError();
}

hipError_t launch_projection_backward(const DeviceWeights& w, const void* z, const uint8_t* mask, int64_t N,
                                      int incoming, const float* dA, const float* dB, const float* dxg, void* dz,
                                      const BackwardBlocks& bb, float* partial, int grid, hipStream_t s) {
    const int64_t units = N * ((N + 31) / 32);
    const float4* p4 = reinterpret_cast<const float4*>(w.proj4);
    const float4* pb = reinterpret_cast<const float4*>(w.projb);
    if (incoming)
        hipLaunchKernelGGL((k_projection_backward<bf16_t, true>), dim3(grid), dim3(256), 0, s, (const bf16_t*)z, mask,
                           (int)N, units, dA, dB, dxg, p4, pb, w.ln_in_w, w.ln_in_b, w.eps, (bf16_t*)dz, bb.dpa,
                           bb.dga, bb.dpb, bb.dgb, bb.xp, partial);
    else
        hipLaunchKernelGGL((k_projection_backward<bf16_t, false>), dim3(grid), dim3(256), 0, s, (const bf16_t*)z, mask,
                           (int)N, units, dA, dB, dxg, p4, pb, w.ln_in_w, w.ln_in_b, w.eps, (bf16_t*)dz, bb.dpa,
                           bb.dga, bb.dpb, bb.dgb, bb.xp, partial);
    return hipGetLastError();
}

hipError_t launch_wgrad(const bf16_t* U, const bf16_t* V, int64_t N, float* partial, int grid, hipStream_t s) {
    const int64_t units = N * ((N + 31) / 32);
    hipLaunchKernelGGL(k_wgrad, dim3(grid), dim3(256), 0, s, U, V, units, partial);
    return hipGetLastError();
}

hipError_t launch_sum_parts(const float* in, int parts, int64_t stride, int n, float* out, hipStream_t s) {
    hipLaunchKernelGGL(k_sum_parts, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, in, parts, stride, n, out);
    return hipGetLastError();
}

}  // namespace trimul
