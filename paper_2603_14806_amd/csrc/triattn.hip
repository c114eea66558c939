// Triangle attention core (Fold-CP, Section 3.2, Eq. 1) on one GPU: for
// row i, head h and query j,
//
//     out_ijh = sum_k softmax_k( q_ijh . k_ikh / sqrt(32) + b_hjk ) v_ikh
//
// over present keys (mask), computed over key chunks with a running maximum
// M, running sum L and unnormalised output A (the ring's tiled softmax:
// each chunk rescales the state by exp(M_old - M_new)).  One call handles
// one key range; the state lives in registers within a call and in caller
// memory between calls.
#include "common.h"
#include "kernels.h"

namespace trimul {
namespace {

constexpr int kHd = 32;          // head dimension
constexpr int kKc = 64;          // keys per chunk
constexpr int kQt = 128;         // queries per work-group (4 waves x 32)
constexpr int kBRow = 68;        // LDS row stride (bf16) of the bias tile [128 q][64 keys]

// K chunk [64 keys][32 d] bf16: 16-byte piece c4 (d = 8 c4 ..) of key kk,
// XOR-swizzled by (kk / 4) % 4 so that 16 keys read start in 16 bank groups.
__device__ __forceinline__ uint32_t koff(int kk, int c4) { return (uint32_t)(kk * 64 + ((c4 ^ ((kk >> 2) & 3)) << 4)); }

__device__ __forceinline__ float xor32(float v) { return __shfl_xor(v, 32); }

// ds_read_b64_tr_b16: in each 16-lane group g, lane 16 g + 4 a + b receives
// element b of the 8-byte chunks addressed by lanes 16 g + a, + 4, + 8, + 12.
typedef short v4i16_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_read_tr4(const void* p) {
    typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;
    return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(p)));
}

struct TaChunk {                 // one chunk's global loads (registers)
    uint4 kv, vv;                // key t / 4, piece t % 4 of K and V
    uint4 bb[4];                 // bias row t / 2, keys 32 (t % 2) .. + 31
    uint32_t m;                  // mask byte of key t (t < 64)
};

template <typename TO>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(3, 3))) void k_triattn(const bf16_t* __restrict__ q, const bf16_t* __restrict__ k,
                                                 const bf16_t* __restrict__ v, const bf16_t* __restrict__ bias,
                                                 const uint8_t* __restrict__ mask, int N, int H, int64_t ldb, int k0,
                                                 int kend,
                                                 float* __restrict__ stA, float* __restrict__ stM,
                                                 float* __restrict__ stL, int load_state, int finish,
                                                 TO* __restrict__ out) {
    __shared__ __align__(16) char ks[2][kKc * 64];            // K chunks
    __shared__ __align__(16) char vs[2][kKc * 64];            // V chunks [64 keys][32 d], row-major
    __shared__ __align__(16) bf16_t bt[2][kQt * kBRow];       // bias tiles
    __shared__ float mb[2][kKc];                              // 0 or -inf per key
    constexpr bool kHiLo = sizeof(TO) == 4;                   // P enters the PV product as hi + lo
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int ql = lane & 31, hi = lane >> 5;
    const int qtiles = (N + kQt - 1) / kQt;
    const int row = blockIdx.x / (H * qtiles);
    const int rem = blockIdx.x - row * H * qtiles;
    const int h = rem / qtiles, j0 = (rem - h * qtiles) * kQt;
    const int j = j0 + 32 * w + ql;                           // this lane's query
    const bool jv = j < N;
    const int64_t rowN = (int64_t)row * N;
    const int nchunks = (kend - k0 + kKc - 1) / kKc;

    // Q^T as the B operand: lane supplies Q[j][16 ks + 8 hi .. + 7]
    bf16x8_t qf[2];
    {
        const auto rq = make_rsrc(q + ((rowN + j0) * H + h) * kHd, (uint32_t)(N - j0) * H * kHd * 2);
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
            qf[s2] = __builtin_bit_cast(bf16x8_t, buf_load16(rq, (uint32_t)(((32 * w + ql) * H) * kHd * 2 + 32 * s2 + 16 * hi)));
    }

    auto load = [&](int c, TaChunk& p) {
        const int kb = k0 + c * kKc;
        const int nk = c < nchunks ? min(kKc, kend - kb) : 0;
        const auto rk = make_rsrc(k + ((rowN + kb) * H + h) * kHd, (uint32_t)nk * H * kHd * 2);
        const auto rv = make_rsrc(v + ((rowN + kb) * H + h) * kHd, (uint32_t)nk * H * kHd * 2);
        const uint32_t ko = (uint32_t)((t >> 2) * H * kHd * 2 + 16 * (t & 3));
        p.kv = buf_load16(rk, ko);                                // keys past the chunk read zero
        p.vv = buf_load16(rv, ko);
        const int br = t >> 1;                                  // bias row j0 + br, keys kb + 32 (t & 1) ..
        const uint32_t rows_ok = (uint32_t)max(0, min(kQt, N - j0));
        // The range check is per dword, so the range ends on a 16-byte boundary
        // (8 keys): a range ending inside a dword would also drop the valid key
        // in it.  Rounding stays within the row (ld_bias % 8 == 0, kb % 8 == 0).
        const auto rb = make_rsrc(bias + ((int64_t)h * N + j0) * ldb + kb,
                                  rows_ok && nk ? (uint32_t)((rows_ok - 1) * ldb + ((nk + 7) & ~7)) * 2 : 0u);
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
            // keys past the chunk read zero or the next keys' bias (never used:
            // those keys carry -inf from the mask row below)
            p.bb[s2] = buf_load16(rb, (uint32_t)(br * ldb * 2 + 64 * (t & 1) + 16 * s2));
        }
        const auto rm = make_rsrc(mask, mask ? (uint32_t)kend : 0u);
        p.m = mask ? __builtin_amdgcn_raw_buffer_load_b8(rm, kb + (t & (kKc - 1)), 0, 0) : 1u;
    };
    auto stage = [&](int c, int buf, const TaChunk& p) {
        const int kb = k0 + c * kKc;
        const int kk = t >> 2, c4 = t & 3;
        *reinterpret_cast<uint4*>(ks[buf] + koff(kk, c4)) = p.kv;
        *reinterpret_cast<uint4*>(vs[buf] + kk * 64 + c4 * 16) = p.vv;   // a wave: 1 KB contiguous
        const int br = t >> 1;
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
            uint2* dst = reinterpret_cast<uint2*>(&bt[buf][br * kBRow + 32 * (t & 1) + 8 * s2]);
            dst[0] = make_uint2(p.bb[s2].x, p.bb[s2].y);
            dst[1] = make_uint2(p.bb[s2].z, p.bb[s2].w);
        }
        if (t < kKc) mb[buf][t] = (kb + t < kend && p.m != 0) ? 0.f : -INFINITY;
    };

    // running state of query j: lanes j and j + 32 hold the same query
    // (different keys / output dims); M is shared, L is split between them
    f32x16_t o;
    float M = -INFINITY, L = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) o[r] = 0.f;
    if (load_state && jv) {
        const int64_t sj = (rowN + j) * H + h;
        const float4* a4 = reinterpret_cast<const float4*>(stA + sj * kHd);
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            const float4 x = a4[2 * a + hi];
            o[4 * a] = x.x; o[4 * a + 1] = x.y; o[4 * a + 2] = x.z; o[4 * a + 3] = x.w;
        }
        const int64_t sm = ((int64_t)row * H + h) * N + j;
        M = stM[sm];
        L = hi ? 0.f : stL[sm];
    }

    const float scale = 0.17677669529663688f;                 // 1 / sqrt(32)
    const int vkey = 4 * (lane >> 5) + ((lane >> 2) & 3);     // transposing reads of V: this lane's key
    const int vdim = 2 * (16 * ((lane >> 4) & 1) + 4 * (lane & 3));   // and byte offset of its 4 dims
    TaChunk cur;
    load(0, cur);
    for (int c = 0; c < nchunks; ++c) {
        const int buf = c & 1;
        stage(c, buf, cur);
        load(c + 1, cur);
        __syncthreads();
        // S^T = K Q^T for the chunk's two 32-key blocks: lane = query, registers = keys
        f32x16_t s[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
#pragma unroll
            for (int r = 0; r < 16; ++r) s[b][r] = 0.f;
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(ks[buf] + koff(32 * b + ql, 2 * s2 + hi));
                s[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[s2], s[b], 0, 0, 0);
            }
        }
        // scale, bias, mask (only a chunk that can hold absent keys: a mask
        // is given, or the chunk runs past the range); chunk maximum
        float cm = -INFINITY;
        const int qrow = 32 * w + ql;
        auto scores = [&](bool masked) {
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    const int kk = 32 * b + 8 * a + 4 * hi;
                    const uint2 bw = *reinterpret_cast<const uint2*>(&bt[buf][qrow * kBRow + kk]);
                    const float bv[4] = {__uint_as_float(bw.x << 16), __uint_as_float(bw.x & 0xffff0000u),
                                         __uint_as_float(bw.y << 16), __uint_as_float(bw.y & 0xffff0000u)};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        float x = s[b][4 * a + e] * scale + bv[e];
                        if (masked) x += mb[buf][kk + e];
                        s[b][4 * a + e] = x;
                        cm = fmaxf(cm, x);
                    }
                }
        };
        if (mask != nullptr || k0 + (c + 1) * kKc > kend) scores(true);
        else scores(false);
        cm = fmaxf(cm, xor32(cm));
        const float Mn = fmaxf(M, cm);
        const bool live = Mn != -INFINITY;                    // some present key so far
        const float alpha = (live && M != -INFINITY) ? __expf(M - Mn) : 0.f;
        // p = exp(x - Mn) = exp2(x log2 e - Mn log2 e), one FMA and one
        // v_exp_f32; with no present key yet the shift is 0 and every x is
        // -inf, so p = 0 without a select
        constexpr float kLog2e = 1.4426950408889634f;
        const float nsh = live ? -Mn * kLog2e : 0.f;
        float ps = 0.f;
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[b][r], kLog2e, nsh));
                s[b][r] = p;
                ps += p;
            }
        L = L * alpha + ps;
#pragma unroll
        for (int r = 0; r < 16; ++r) o[r] *= alpha;
        M = Mn;
        // O^T += V^T P^T: k-step (b, t2) covers keys 32 b + 16 t2 .. + 15; half hi supplies keys
        // {16 t2 + 4 hi + 0..3, 16 t2 + 8 + 4 hi + 0..3} = registers 8 t2 .. 8 t2 + 7.  The V^T
        // fragment (lane: output dim ql, those 8 keys) comes from the row-major V chunk through two
        // transposing reads: addressing lane 16 g + 4 i + a points at key 4 (g >> 1) + i (+ 8 for
        // the second read) and dims 16 (g & 1) + 4 a .. + 3, so lane l receives dim l % 32 of four
        // consecutive keys.
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                const char* vr = vs[buf] + (32 * b + 16 * t2 + vkey) * 64 + vdim;
                const uint2 v0 = lds_read_tr4(vr);
                const uint2 v1 = lds_read_tr4(vr + 8 * 64);
                const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, make_uint4(v0.x, v0.y, v1.x, v1.y));
                // P as bf16 hi + lo for fp32 output (~16 mantissa bits of p); with
                // bf16 output the hi part alone (its 2^-9 rounding averages over the
                // keys, below the output's own rounding)
                uint32_t ph[4], pl[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float x0 = s[b][8 * t2 + 2 * e], x1 = s[b][8 * t2 + 2 * e + 1];
                    ph[e] = pack_bf16x2(x0, x1);
                    if constexpr (kHiLo)
                        pl[e] = pack_bf16x2(x0 - __uint_as_float(ph[e] << 16), x1 - __uint_as_float(ph[e] & 0xffff0000u));
                }
                o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, __builtin_bit_cast(bf16x8_t, make_uint4(ph[0], ph[1], ph[2], ph[3])), o, 0, 0, 0);
                if constexpr (kHiLo)
                    o = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, __builtin_bit_cast(bf16x8_t, make_uint4(pl[0], pl[1], pl[2], pl[3])), o, 0, 0, 0);
            }
        // no barrier here: the next chunk stages into the other buffer, and the
        // one after that only once every wave has passed the next barrier
    }

    // lane holds output dims d = 8 a + 4 hi + 0..3 of query j
    const float Lt = L + xor32(L);
    if (!jv) return;
    const int64_t sj = (rowN + j) * H + h;
    if (finish) {
        const float inv = Lt > 0.f ? 1.f / Lt : 0.f;
        TO* dst = out + sj * kHd;
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            const int d = 8 * a + 4 * hi;
            if constexpr (sizeof(TO) == 4) {
                *reinterpret_cast<float4*>(dst + d) =
                    make_float4(o[4 * a] * inv, o[4 * a + 1] * inv, o[4 * a + 2] * inv, o[4 * a + 3] * inv);
            } else {
                *reinterpret_cast<uint2*>(dst + d) = make_uint2(pack_bf16x2(o[4 * a] * inv, o[4 * a + 1] * inv),
                                                                pack_bf16x2(o[4 * a + 2] * inv, o[4 * a + 3] * inv));
            }
        }
    } else {
        float4* a4 = reinterpret_cast<float4*>(stA + sj * kHd);
#pragma unroll
        for (int a = 0; a < 4; ++a) a4[2 * a + hi] = make_float4(o[4 * a], o[4 * a + 1], o[4 * a + 2], o[4 * a + 3]);
        if (!hi) {
            const int64_t sm = ((int64_t)row * H + h) * N + j;
            stM[sm] = M;
            stL[sm] = Lt;
        }
    }
}

}  // namespace

hipError_t launch_triattn(int out_dtype, const void* q, const void* k, const void* v, const void* bias,
                          const uint8_t* mask, int64_t rows, int64_t N, int H, int64_t ldb, int64_t k0, int64_t kend,
                          float* stA,
                          float* stM, float* stL, int load_state, int finish, void* out, hipStream_t s) {
    const int64_t grid = rows * H * ((N + kQt - 1) / kQt);
    if (out_dtype == 0)
        hipLaunchKernelGGL(k_triattn<float>, dim3((unsigned)grid), dim3(256), 0, s, (const bf16_t*)q, (const bf16_t*)k,
                           (const bf16_t*)v, (const bf16_t*)bias, mask, (int)N, H, ldb, (int)k0, (int)kend, stA, stM, stL,
                           load_state, finish, (float*)out);
    else
        hipLaunchKernelGGL(k_triattn<bf16_t>, dim3((unsigned)grid), dim3(256), 0, s, (const bf16_t*)q,
                           (const bf16_t*)k, (const bf16_t*)v, (const bf16_t*)bias, mask, (int)N, H, ldb, (int)k0,
                           (int)kend, stA, stM, stL, load_state, finish, (bf16_t*)out);
    return hipGetLastError();
}

}  // namespace trimul
