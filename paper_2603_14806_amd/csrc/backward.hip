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
