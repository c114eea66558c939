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

    for (int idx = t; idx < kPairs * kCh; idx += 256) {
        const int c = idx / kPairs, p = idx % kPairs;
        cs[p][c] = p < np ? a.C[c * a.sc + i * a.ldc + j0 + p] : 0.f;
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
        s1 += __shfl_xor(s1, 1);
        s1 += __shfl_xor(s1, 2);
        s2 += __shfl_xor(s2, 1);
        s2 += __shfl_xor(s2, 2);
        const float mu1 = s1 * (1.0f / kCh), mu2 = s2 * (1.0f / kCz);
        float v1 = 0.f, v2 = 0.f;
        for (int d = q * 32; d < q * 32 + 32; ++d) {
            const float e1 = cs[p][d] - mu1, e2 = xs[p][d] - mu2;
            v1 += e1 * e1;
            v2 += e2 * e2;
        }
        v1 += __shfl_xor(v1, 1);
        v1 += __shfl_xor(v1, 2);
        v2 += __shfl_xor(v2, 1);
        v2 += __shfl_xor(v2, 2);
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

template <typename T, typename TO>
hipError_t launch_valu(const DeviceWeights& w, const EpilogueArgs& a, hipStream_t s) {
    const int64_t nchunk = (a.cols + kPairs - 1) / kPairs;
    hipLaunchKernelGGL((k3_epilogue_valu<T, TO>), dim3((unsigned)(a.rows * nchunk)), dim3(256), 0, s, a,
                       nchunk, w.wo_t, w.wg_t, w.ln_in_w, w.ln_in_b, w.ln_out_w, w.ln_out_b, w.eps);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_epilogue(int dtype, int out_dtype, const DeviceWeights& w, const EpilogueArgs& a,
                           hipStream_t s) {
    if (dtype == 0)
        return out_dtype == 0 ? launch_valu<float, float>(w, a, s) : launch_valu<float, bf16_t>(w, a, s);
    return out_dtype == 0 ? launch_valu<bf16_t, float>(w, a, s) : launch_valu<bf16_t, bf16_t>(w, a, s);
}

}  // namespace trimul
