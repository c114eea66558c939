// Outer product mean (Fold-CP, Section 3.5) on one GPU: the layout kernel
// that turns one step's sequences into operands of the contraction, and the
// projection epilogue.  The sum over sequences itself,
//
//     O[(i, c)][(j, d)] = sum_s m_si m_sj a_sic b_sjd,
//
// is one NT product with M = rows * D, N = cols * D, K = slen (both operands
// given transposed, which is the input's own order), and the pair
// counts n_ij = sum_s m_si m_sj another with M = rows, N = cols (0/1
// operands: exact in fp32 up to 2^24); both run on the contraction kernel
// (k2_contract_ws), accumulating over the steps of a tile.
#include "common.h"
#include "kernels.h"

namespace trimul {
namespace {

constexpr int kD = 32;         // channels of a and b
constexpr int kOz = 128;       // output channels

// ---------------------------------------------------------------- pack
//
// The sums' operands are given to the contraction transposed: X[s][(tok, c)]
// = m_s,tok a_s,tok,c in the panel layout of slen rows and ntok * 32 columns,
// where the 32-column block of token tok and the 256-row block of sequences
// s / 256 is one contiguous 16 KB block holding, for each sequence, the 64
// bytes a[s][tok][0:32] as they are in the input.  So the pack is a masked
// copy, no transpose.  One work-group per (8 tokens, 32 sequences): thread t
// takes token part t % 8 (eight consecutive tokens of one sequence read 512
// contiguous bytes) and sequence t / 8 (the eight sequences of a wave and
// token write 512 contiguous bytes).  Sequences from slen up to the panel's
// 256-row boundary get zeros; tokens past ntok have no columns and write
// nothing.  The pair counts' operands keep the plain blocked layout (row =
// token, k = s, bf16 0/1), written for k below the panel's 32-step boundary.
__global__ __launch_bounds__(256) void k_opm_pack(const bf16_t* __restrict__ a, const uint8_t* __restrict__ mask,
                                                  int64_t n_total, int64_t tok0, int ntok, int64_t s0, int slen,
                                                  bf16_t* __restrict__ P, bf16_t* __restrict__ Mp) {
    const int t = threadIdx.x;
    const int part = t & 7, sl = t >> 3;
    const int tok = blockIdx.y * 8 + part, s = blockIdx.x * 32 + sl;
    uint4 v[4] = {};
    bf16_t m = 0;
    if (tok < ntok && s < slen) {
        const int64_t src = ((s0 + s) * n_total + tok0 + tok);
        const uint8_t mk = mask ? mask[src] : (uint8_t)1;
        if (mk) {
            const uint4* p = reinterpret_cast<const uint4*>(a + src * kD);
#pragma unroll
            for (int q = 0; q < 4; ++q) v[q] = p[q];
            m = 0x3f80;   // bf16 1.0
        }
    }
    if (tok < ntok) {
        const PanelGeom xg = panel_geom(slen, (int64_t)ntok * kD);
        uint4* dst = reinterpret_cast<uint4*>(P + panel_off(xg, 0, s, (int64_t)tok * kD));
#pragma unroll
        for (int q = 0; q < 4; ++q) dst[q] = v[q];
    }
    const PanelGeom mg = panel_geom(ntok, slen);
    if (s < mg.ksteps * 32) Mp[panel_off(mg, 0, tok, s)] = m;
}

// ---------------------------------------------------------------- epilogue
//
// out_ij[e] = (1 / n_ij) sum_{c,d} W_o[e][c * 32 + d] O[(i, c)][(j, d)] + b_o[e]
// (the sum is 0 where n_ij = 0), on matrix cores (v_mfma_f32_16x16x32_bf16):
// unit = 32 pairs (i, j0 .. j0 + 31); the k dimension of the product runs
// over (c, d), one k-step per c.  8 waves, wave w owns output channels
// 16 w .. 16 w + 15 and keeps its W_o rows in registers (32 x bf16x8); the
// unit's sums (32 rows c x 1024 floats) go through LDS in four chunks of 8
// rows, double-buffered, as bf16 hi + lo (so the product carries ~16
// mantissa bits of the fp32 sums).  Operand layout: lane l supplies row
// (column) l % 16 and k values 8 (l / 16) .. + 7; the result gives lane l
// column l % 16 and rows 4 (l / 16) + 0 .. 3.
constexpr int kEt = 512;
constexpr int kChunk = 8;                          // rows c per LDS chunk
constexpr int kCkBytes = kChunk * 32 * 64;         // bf16 [8 c][32 pairs][32 d] = 16 KB
constexpr int kOrow = kOz + 4;                     // output staging row stride (floats)

// Byte offset of the 16-byte piece kq (d = 8 kq .. + 7) of pair p, row c of a
// chunk: rows of 64 bytes, pieces XOR-swizzled by (p / 4) % 4 so that the 16
// pairs of an operand read start in 16 different bank groups.
__device__ __forceinline__ uint32_t ck_off(int c, int p, int kq) {
    return (uint32_t)((c * 32 + p) * 64 + ((kq ^ ((p >> 2) & 3)) << 4));
}

template <typename TO>
__global__ __launch_bounds__(kEt) void k_opm_epilogue(const float* __restrict__ O, const float* __restrict__ cnt,
                                                     int rows, int cols, int64_t ldo, int64_t ldc,
                                                     const bf16_t* __restrict__ wo, const float* __restrict__ bo,
                                                     TO* __restrict__ out) {
    __shared__ __align__(16) char ck[2][2][kCkBytes];     // [buffer][hi, lo]
    __shared__ __align__(16) float os[32 * kOrow];       // outputs [pair][e]
    __shared__ float ns[32];                             // 1 / n of the unit's pairs (0 where n = 0)
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int col = lane & 15, kq = lane >> 4;
    const int J = (cols + 31) / 32;
    const int64_t units = (int64_t)rows * J;

    bf16x8_t wr[32];                                     // W_o[16 w + col][c * 32 + 8 kq ..]
#pragma unroll
    for (int c = 0; c < 32; ++c)
        wr[c] = *reinterpret_cast<const bf16x8_t*>(wo + (int64_t)(16 * w + col) * (kD * kD) + c * kD + 8 * kq);
    const float bias = bo[16 * w + col];
    wait_vmcnt<0>();

    // staging of chunk q of unit u: thread t moves row c = 8 q + t / 64,
    // floats 16 (t % 64) .. + 15 of the unit's 1024 (pair (t % 64) / 2,
    // d = 16 (t % 2) .. + 15); past the last column the loads read zero.
    auto load = [&](int64_t u, int q, float4 (&v)[4]) {
        const bool valid = u < units;
        const int64_t uu = valid ? u : 0;
        const int i = (int)(uu / J), j0 = (int)(uu - (int64_t)i * J) * 32;
        const int c = kChunk * q + (t >> 6);
        const uint32_t bytes = valid ? (uint32_t)(cols - j0) * kD * 4 : 0u;
        const auto r = make_rsrc(O + ((int64_t)i * kD + c) * ldo + (int64_t)j0 * kD, bytes);
#pragma unroll
        for (int k = 0; k < 4; ++k)
            v[k] = __builtin_bit_cast(float4, buf_load16(r, (uint32_t)(64 * (t & 63) + 16 * k)));
    };
    auto stage = [&](int buf, const float4 (&v)[4]) {
        const int cl = t >> 6, p = (t & 63) >> 1, h = t & 1;
        const float f[16] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w,
                             v[2].x, v[2].y, v[2].z, v[2].w, v[3].x, v[3].y, v[3].z, v[3].w};
#pragma unroll
        for (int g = 0; g < 2; ++g) {
            uint32_t hw[4], lw[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float x0 = f[8 * g + 2 * k], x1 = f[8 * g + 2 * k + 1];
                hw[k] = pack_bf16x2(x0, x1);
                lw[k] = pack_bf16x2(x0 - __uint_as_float(hw[k] << 16), x1 - __uint_as_float(hw[k] & 0xffff0000u));
            }
            const uint32_t off = ck_off(cl, p, 2 * h + g);
            *reinterpret_cast<uint4*>(ck[buf][0] + off) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
            *reinterpret_cast<uint4*>(ck[buf][1] + off) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
        }
    };

    float4 v[4];
    int64_t u = blockIdx.x;
    load(u, 0, v);
    f32x4_t acc[2];
    for (; u < units; u += gridDim.x) {
        const int i = (int)(u / J), j0 = (int)(u - (int64_t)i * J) * 32;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        if (t < 32) {
            const float n = (j0 + t < cols) ? cnt[(int64_t)i * ldc + j0 + t] : 0.f;
            ns[t] = n > 0.f ? 1.f / n : 0.f;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int buf = q & 1;
            stage(buf, v);
            if (q < 3) load(u, q + 1, v);
            else load(u + gridDim.x, 0, v);
            __syncthreads();
#pragma unroll
            for (int cl = 0; cl < kChunk; ++cl)
#pragma unroll
                for (int mb = 0; mb < 2; ++mb) {
                    const uint32_t off = ck_off(cl, 16 * mb + col, kq);
                    const bf16x8_t xh = *reinterpret_cast<const bf16x8_t*>(ck[buf][0] + off);
                    const bf16x8_t xl = *reinterpret_cast<const bf16x8_t*>(ck[buf][1] + off);
                    acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xh, wr[kChunk * q + cl], acc[mb], 0, 0, 0);
                    acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xl, wr[kChunk * q + cl], acc[mb], 0, 0, 0);
                }
        }
        // lane holds channel e = 16 w + col of pairs 16 mb + 4 kq + r
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int p = 16 * mb + 4 * kq + r;
                os[p * kOrow + 16 * w + col] = acc[mb][r] * ns[p] + bias;
            }
        __syncthreads();
        {   // 32 pairs x 128 channels, contiguous in out: 16-byte stores, pairs past cols dropped
            const auto ro = make_rsrc(out + ((int64_t)i * cols + j0) * kOz, (uint32_t)(cols - j0) * kOz * sizeof(TO));
            if constexpr (sizeof(TO) == 4) {
#pragma unroll
                for (int k = 0; k < 2; ++k) {
                    const int e4 = t + kEt * k, p = e4 >> 5, e = 4 * (e4 & 31);
                    const float4 f = *reinterpret_cast<const float4*>(&os[p * kOrow + e]);
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i_t, f), ro, (p * kOz + e) * 4, 0, 0);
                }
            } else {
                const int p = t >> 4, e = 8 * (t & 15);
                const float4 f0 = *reinterpret_cast<const float4*>(&os[p * kOrow + e]);
                const float4 f1 = *reinterpret_cast<const float4*>(&os[p * kOrow + e + 4]);
                const uint4 pk = make_uint4(pack_bf16x2(f0.x, f0.y), pack_bf16x2(f0.z, f0.w), pack_bf16x2(f1.x, f1.y),
                                            pack_bf16x2(f1.z, f1.w));
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4i_t, pk), ro, (p * kOz + e) * 2, 0, 0);
            }
        }
        // os and ns are rewritten by the next unit only after its first barrier
    }
}

}  // namespace

hipError_t launch_opm_pack(const void* a, const uint8_t* mask, int64_t n_total, int64_t tok0, int64_t ntok,
                           int64_t s0, int64_t slen, void* P, void* Mp, hipStream_t s) {
    const dim3 grid((unsigned)((slen + 255) / 256 * 8), (unsigned)((ntok + 7) / 8));
    hipLaunchKernelGGL(k_opm_pack, grid, dim3(256), 0, s, (const bf16_t*)a, mask, n_total, tok0, (int)ntok, s0,
                       (int)slen, (bf16_t*)P, (bf16_t*)Mp);
    return hipGetLastError();
}

hipError_t launch_opm_epilogue(int out_dtype, const float* O, const float* cnt, int64_t rows, int64_t cols,
                               const uint16_t* wo, const float* bo, void* out, int cus, hipStream_t s) {
    const int64_t units = rows * ((cols + 31) / 32);
    const unsigned g = (unsigned)(units < cus ? units : cus);
    const int64_t ldo = cols * kD, ldc = (cols + 31) / 32 * 32;
    if (out_dtype == 0)
        hipLaunchKernelGGL(k_opm_epilogue<float>, dim3(g), dim3(kEt), 0, s, O, cnt, (int)rows, (int)cols, ldo, ldc,
                           (const bf16_t*)wo, bo, (float*)out);
    else
        hipLaunchKernelGGL(k_opm_epilogue<bf16_t>, dim3(g), dim3(kEt), 0, s, O, cnt, (int)rows, (int)cols, ldo, ldc,
                           (const bf16_t*)wo, bo, (bf16_t*)out);
    return hipGetLastError();
}

}  // namespace trimul
