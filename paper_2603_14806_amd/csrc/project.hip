// K1: input LayerNorm + gated a/b projections + pair mask, writing the
// channel-major operands of the contraction (Section 3.3: a, b are gated
// projections of z; Eq. 2 / Eq. 3 pick which token index is contracted).
//
// Work unit: a "line" of 64 pairs that share one output row.  Outgoing line
// (r, k0): pairs (r, k0..k0+63), A[c][r][k0+p] = a(r, k0+p).  Incoming line
// (r, k0): pairs (k0..k0+63, r), A[c][r][k0+p] = a(k0+p, r).  Either way the
// 64 results of one channel are contiguous in A and B.
#include "common.h"
#include "kernels.h"

namespace trimul {
namespace {

constexpr int kLine = 64;   // pairs per work unit

// Scalar (VALU) fp32 version; it serves the fp32 storage path.
template <typename T, bool INCOMING>
__global__ __launch_bounds__(256) void k1_project_valu(
    const T* __restrict__ z, const uint8_t* __restrict__ mask, int64_t N, int64_t ld, int64_t nchunk,
    const float4* __restrict__ proj4, const float* __restrict__ lnw, const float* __restrict__ lnb,
    float eps, T* __restrict__ A, T* __restrict__ B) {
    __shared__ float xs[kLine][kCz + 1];
    const int t = threadIdx.x;
    const int64_t r = blockIdx.x / nchunk;
    const int64_t k0 = (blockIdx.x % nchunk) * kLine;
    const int np = (int)min<int64_t>(kLine, N - k0);

    for (int idx = t; idx < kLine * kCz; idx += 256) {
        const int p = idx / kCz, d = idx % kCz;
        float v = 0.f;
        if (p < np) {
            const int64_t pair = INCOMING ? (k0 + p) * N + r : r * N + k0 + p;
            v = Store<T>::ld(z + pair * kCz + d);
        }
        xs[p][d] = v;
    }
    __syncthreads();

    {   // LayerNorm over c_z, four lanes per pair
        const int p = t >> 2, q = t & 3;
        float s = 0.f;
        for (int d = q * 32; d < q * 32 + 32; ++d) s += xs[p][d];
        s += __shfl_xor(s, 1);
        s += __shfl_xor(s, 2);
        const float mu = s * (1.0f / kCz);
        float v = 0.f;
        for (int d = q * 32; d < q * 32 + 32; ++d) {
            const float e = xs[p][d] - mu;
            v += e * e;
        }
        v += __shfl_xor(v, 1);
        v += __shfl_xor(v, 2);
        const float rs = rsqrtf(v * (1.0f / kCz) + eps);
        for (int d = q * 32; d < q * 32 + 32; ++d) xs[p][d] = (xs[p][d] - mu) * rs * lnw[d] + lnb[d];
    }
    __syncthreads();

    const int c = t & (kCh - 1), half = t >> 7;
    float acc[32][4];
#pragma unroll
    for (int q = 0; q < 32; ++q) acc[q][0] = acc[q][1] = acc[q][2] = acc[q][3] = 0.f;
    for (int d = 0; d < kCz; ++d) {
        const float4 w = proj4[d * kCh + c];
#pragma unroll
        for (int q = 0; q < 32; ++q) {
            const float x = xs[half * 32 + q][d];
            acc[q][0] += w.x * x;
            acc[q][1] += w.y * x;
            acc[q][2] += w.z * x;
            acc[q][3] += w.w * x;
        }
    }
    const bool mr = mask ? mask[r] != 0 : true;
#pragma unroll
    for (int q = 0; q < 32; ++q) {
        const int p = half * 32 + q;
        if (p < np) {
            const bool m = mr && (mask ? mask[k0 + p] != 0 : true);
            const float a = m ? sigmoidf_(acc[q][1]) * acc[q][0] : 0.f;
            const float b = m ? sigmoidf_(acc[q][3]) * acc[q][2] : 0.f;
            const int64_t off = ((int64_t)c * N + r) * ld + k0 + p;
            Store<T>::st(A + off, a);
            Store<T>::st(B + off, b);
        }
    }
}

}  // namespace

hipError_t launch_project(int dtype, const DeviceWeights& w, const void* z, const uint8_t* mask,
                          int64_t N, int64_t ld, int incoming, void* A, void* B, hipStream_t s) {
    const int64_t nchunk = (N + kLine - 1) / kLine;
    const dim3 grid((unsigned)(N * nchunk)), block(256);
    const float4* p4 = reinterpret_cast<const float4*>(w.proj4);
    if (dtype == 0) {
        if (incoming)
            hipLaunchKernelGGL((k1_project_valu<float, true>), grid, block, 0, s, (const float*)z, mask, N,
                               ld, nchunk, p4, w.ln_in_w, w.ln_in_b, w.eps, (float*)A, (float*)B);
        else
            hipLaunchKernelGGL((k1_project_valu<float, false>), grid, block, 0, s, (const float*)z, mask, N,
                               ld, nchunk, p4, w.ln_in_w, w.ln_in_b, w.eps, (float*)A, (float*)B);
    } else {
        if (incoming)
            hipLaunchKernelGGL((k1_project_valu<bf16_t, true>), grid, block, 0, s, (const bf16_t*)z, mask, N,
                               ld, nchunk, p4, w.ln_in_w, w.ln_in_b, w.eps, (bf16_t*)A, (bf16_t*)B);
        else
            hipLaunchKernelGGL((k1_project_valu<bf16_t, false>), grid, block, 0, s, (const bf16_t*)z, mask, N,
                               ld, nchunk, p4, w.ln_in_w, w.ln_in_b, w.eps, (bf16_t*)A, (bf16_t*)B);
    }
    return hipGetLastError();
}

}  // namespace trimul
