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
// (c, i, j) -> X_c[i][k = j], converted to T.  One unit = two rows i, i + 1
// (i even) and one 32-column block: 2 x 128 channels x 32 floats, contiguous
// per channel in the result layout; in the panel the two rows of a channel
// are adjacent (one 128-byte line in bf16), so no store writes a partial
// line.  Thread t moves channel t / 2, columns 16 (t % 2) .. + 15 of both
// rows.  Columns past N carry whatever the result layout holds there into
// the k padding of the panel, which the contraction never uses.
template <typename T>
__global__ __launch_bounds__(256) void k_result_to_panel(const float* __restrict__ R, T* __restrict__ P, int N,
                                                        int64_t units) {
    const int t = threadIdx.x, ch = t >> 1, h = t & 1;
    const int J = (N + kResJ - 1) / kResJ;
    const PanelGeom pg = panel_geom(N, N);
    for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
        const int64_t ip = u / J, jb = u - (u / J) * J;
        const int64_t i0 = 2 * ip;
        const int nr = i0 + 1 < N ? 2 : 1;                 // an odd N's last unit holds one row
        float4 v[2][4];
#pragma unroll
        for (int rr = 0; rr < 2; ++rr) {
            if (rr < nr) {
                const float4* src = reinterpret_cast<const float4*>(R + result_off(J, kCh, ch, i0 + rr, jb * kResJ) + 16 * h);
#pragma unroll
                for (int q = 0; q < 4; ++q) v[rr][q] = src[q];
            }
        }
#pragma unroll
        for (int rr = 0; rr < 2; ++rr) {
            if (rr >= nr) break;
            T* dst = P + panel_off(pg, ch, i0 + rr, jb * kResJ + 16 * h);
            if constexpr (sizeof(T) == 2) {
                uint4 o[2];
                o[0] = make_uint4(pack_bf16x2(v[rr][0].x, v[rr][0].y), pack_bf16x2(v[rr][0].z, v[rr][0].w),
                                  pack_bf16x2(v[rr][1].x, v[rr][1].y), pack_bf16x2(v[rr][1].z, v[rr][1].w));
                o[1] = make_uint4(pack_bf16x2(v[rr][2].x, v[rr][2].y), pack_bf16x2(v[rr][2].z, v[rr][2].w),
                                  pack_bf16x2(v[rr][3].x, v[rr][3].y), pack_bf16x2(v[rr][3].z, v[rr][3].w));
                reinterpret_cast<uint4*>(dst)[0] = o[0];
                reinterpret_cast<uint4*>(dst)[1] = o[1];
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q) reinterpret_cast<float4*>(dst)[q] = v[rr][q];
            }
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
// block [128 channels][32 slots] at u * 4096 elements.  Each weight gradient
// is then a sum over units of U_block * V_block^T (k_wgrad); slots of pairs
// past N or masked out carry a zero in at least one of the two blocks.
//
// The per-pair stages are 128-wide products per unit, run on matrix cores
// (v_mfma_f32_16x16x32_bf16): 8 waves, wave w owns the 16 output columns
// 16 w .. 16 w + 15 of every product and keeps its slice of the weights in
// VGPRs as the B operand.  Activations are the A operand, split into
// bf16 hi + lo (two products), so the products carry about 16 mantissa bits
// of the fp32 activations; the weights are bf16 already.  Operand layout of
// the 16 x 16 x 32 product: lane l supplies row (or column) l % 16 and the
// eight k values 8 (l / 16) .. + 7; the result gives lane l column l % 16 and
// rows 4 (l / 16) + 0 .. 3.
constexpr int kQ = 32;        // pairs per unit
constexpr int kBT = 512;      // threads of the per-pair backward kernels
constexpr int kCs = 36;       // row stride (floats) of [channel][pair] tiles
constexpr int kPq = 148;      // row stride (floats) of [pair][channel] tiles (the fewest bank conflicts
                              // over their four access patterns)
constexpr int kArow = 256;    // bytes of one bf16 activation row [128]

// Byte offset of 16-byte chunk ch of row p in a bf16 [q][128] tile; chunks
// are XOR-swizzled over 16 rows so that the A-operand reads (16 rows, one
// chunk each) hit distinct banks.
__device__ __forceinline__ uint32_t arow(int p, int ch) { return (uint32_t)(p * kArow + ((ch ^ (p & 15)) << 4)); }

// The value itself, hidden from the optimiser: lane indices passed through
// this inside a loop make the LDS addresses derived from them loop-variant,
// so they are recomputed where used instead of being hoisted out of the loop
// and held in (or spilled from) registers for the whole kernel.
__device__ __forceinline__ int opaque(int v) {
    asm volatile("" : "+v"(v));
    return v;
}

__device__ __forceinline__ float sum_lanes16(float v) {
    v = sum_lanes8(v);
    v += dpp_mov<0x140>(v);   // row_mirror: lane i meets lane 15 - i (the other group of 8)
    return v;
}

__device__ __forceinline__ void st_hilo(char* hi, char* lo, uint32_t off, float v) {
    const bf16_t h = f2bf(v);
    *reinterpret_cast<bf16_t*>(hi + off) = h;
    *reinterpret_cast<bf16_t*>(lo + off) = f2bf(v - bf2f(h));
}

__device__ __forceinline__ f32x4_t mfma16(bf16x8_t a, bf16x8_t b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8_t ld_frag(const char* base, uint32_t off) {
    return *reinterpret_cast<const bf16x8_t*>(base + off);
}

// Range-checked buffer access (make_rsrc): loads past the resource's size
// read zero and stores past it are dropped, so tails need no branches and
// every pass of a unit loop issues the same memory instructions (which keeps
// the compiler's wait counts exact).
__device__ __forceinline__ float4 bld_f4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(float4, buf_load16(r, off));
}
__device__ __forceinline__ uint32_t bld_u8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b8(r, (int)off, 0, 0);
}
__device__ __forceinline__ void bst_f32(__amdgpu_buffer_rsrc_t r, uint32_t off, float v) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)off, 0, 0);
}
__device__ __forceinline__ void bst_u4(__amdgpu_buffer_rsrc_t r, uint32_t off, uint4 v) {
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, (int)off, 0, 0);
}

// 8 bf16 of column `col` of a swizzled row tile, rows q0 .. q0 + 7, packed.
__device__ __forceinline__ uint4 gather_col8(const char* tile, int q0, int col) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int q = q0 + 2 * i;
        const uint32_t a = *reinterpret_cast<const bf16_t*>(tile + arow(q, col >> 3) + 2 * (col & 7));
        const uint32_t b = *reinterpret_cast<const bf16_t*>(tile + arow(q + 1, col >> 3) + 2 * (col & 7));
        w[i] = a | (b << 16);
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

// Four bf16 (rows 4 kq .. + 3 of one 16 x 16 result tile) as one 8-byte word.
__device__ __forceinline__ uint2 pack4(float a, float b, float c, float d) {
    return make_uint2(pack_bf16x2(a, b), pack_bf16x2(c, d));
}

template <typename TO> struct DoutRegs;
template <> struct DoutRegs<float> { float4 a, b; };
template <> struct DoutRegs<bf16_t> { uint4 a; };

// Epilogue backward.  For the unit's pairs (r, k): recompute x = LN_in(z),
// y = LN_out(C), u = W_o y, g = sigmoid(W_g x); then
//   du = dout m g,  dgg = dout m u g (1 - g),  dy = du W_o,  dx_g = dgg W_g,
//   dC = LN_out backward of dy.
// Writes dC into the panel (row r, columns k), dx_g [pair][c_z] fp32, unit
// blocks du, y, dgg, x, and per-work-group sums of dgamma_out, dbeta_out at
// partial[(2 wg + {0, 1}) * 128 + c].
template <typename TO>
__global__ __launch_bounds__(kBT) void k_epilogue_backward(
    const float* __restrict__ C, const bf16_t* __restrict__ z, const uint8_t* __restrict__ mask,
    const TO* __restrict__ dout, int N, int64_t units, const bf16_t* __restrict__ wfwd,
    const bf16_t* __restrict__ wbwd, const float* __restrict__ lniw, const float* __restrict__ lnib,
    const float* __restrict__ lnow, const float* __restrict__ lnob, float eps, bf16_t* __restrict__ dCp,
    float* __restrict__ dxg, bf16_t* __restrict__ b_du, bf16_t* __restrict__ b_y, bf16_t* __restrict__ b_dgg,
    bf16_t* __restrict__ b_x, float* __restrict__ partial) {
    __shared__ __align__(16) float cs[kCh * kCs];        // C [c][q]
    __shared__ __align__(16) float dq[kQ * kPq];         // dout [q][d], then dy [q][c]
    __shared__ __align__(16) float dct[kCh * kCs];       // dC [c][q]
    __shared__ __align__(16) char act[4][kQ * kArow];    // y hi, y lo, x hi, x lo  [q][128]
    __shared__ __align__(16) char act2[4][kQ * kArow];   // du hi, du lo, dgg hi, dgg lo  [q][128]
    // gamma_out, beta_out, gamma_in, beta_in; rows 2 and 3 put channel d at
    // d + 4 (d / 64), so that the 16 addresses 8 l + 2 i of a LayerNorm-input
    // read fall in distinct banks
    __shared__ float prm[4][136];
    __shared__ float mq[kQ];                             // pair mask of the unit
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int lp = t >> 4, lq = t & 15;                  // LayerNorms: pair lp, 16 lanes per pair
    const int col = lane & 15, kq = lane >> 4;           // MFMA operand / result lanes
    const int sc = t >> 2, sq = t & 3;                   // channel-major stores: channel sc, pairs 8 sq .. + 7
    const int J = (N + kQ - 1) / kQ;
    const PanelGeom pg = panel_geom(N, N);

    // Global loads of one unit, issued one unit ahead into the registers the
    // current unit has just released; nothing here reads the loaded
    // registers, so the loads stay in flight until the unit starts.
    struct Pre {
        float4 c0, c1;        // C block floats 4 t .. and 2048 + 4 t ..
        uint4 zv;             // z of pair lp, channels 8 lq .. + 7
        DoutRegs<TO> o;       // dout of pair lp, channels 8 lq .. + 7
        uint32_t mr, mk;      // mask bytes of row r and of column k0 + t % 32 (zero past N)
    };
    auto load = [&](int64_t u, Pre& p) {
        const bool valid = u < units;                     // past the end: zero-size resources
        const int64_t uu = valid ? u : 0;
        const int r = (int)(uu / J), k0 = (int)(uu - (int64_t)r * J) * kQ;
        const int np = min(kQ, N - k0);
        const int64_t pr0 = (int64_t)r * N + k0;          // the unit's first pair
        const auto rc = make_rsrc(C + uu * (kCh * kQ), valid ? kCh * kQ * 4 : 0);
        p.c0 = bld_f4(rc, 16 * t);
        p.c1 = bld_f4(rc, 16 * (t + kBT));
        const auto rzr = make_rsrc(z + pr0 * kCz, valid ? np * kCz * 2 : 0);
        p.zv = buf_load16(rzr, lp * kCz * 2 + 16 * lq);
        if constexpr (sizeof(TO) == 4) {
            const auto ro = make_rsrc(dout + pr0 * kCz, valid ? np * kCz * 4 : 0);
            p.o.a = bld_f4(ro, lp * kCz * 4 + 32 * lq);
            p.o.b = bld_f4(ro, lp * kCz * 4 + 32 * lq + 16);
        } else {
            const auto ro = make_rsrc(dout + pr0 * kCz, valid ? np * kCz * 2 : 0);
            p.o.a = buf_load16(ro, lp * kCz * 2 + 16 * lq);
        }
        const auto rm = make_rsrc(mask, (valid && mask) ? (uint32_t)N : 0u);
        p.mr = bld_u8(rm, opaque(r));                    // per lane: a uniform load would be waited for at once
        p.mk = bld_u8(rm, k0 + (t & (kQ - 1)));
    };

    float accg[8], accb[8];                              // dgamma_out, dbeta_out of c = lq + 16 i
#pragma unroll
    for (int i = 0; i < 8; ++i) accg[i] = accb[i] = 0.f;
    Pre cur;
    load(blockIdx.x, cur);
    bf16x8_t wo[4], wg[4], wot[4], wgt[4];               // B operands: W_o, W_g rows n; W_o^T, W_g^T rows n
    {
        const int n = 16 * w + col;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int k = 32 * ks + 8 * kq;
            wo[ks] = *reinterpret_cast<const bf16x8_t*>(wfwd + n * 128 + k);
            wg[ks] = *reinterpret_cast<const bf16x8_t*>(wfwd + (128 + n) * 128 + k);
            wot[ks] = *reinterpret_cast<const bf16x8_t*>(wbwd + n * 128 + k);
            wgt[ks] = *reinterpret_cast<const bf16x8_t*>(wbwd + (128 + n) * 128 + k);
        }
    }
    if (t < 128) {
        prm[0][t] = lnow[t];
        prm[1][t] = lnob[t];
        prm[2][t + 4 * (t >> 6)] = lniw[t];
        prm[3][t + 4 * (t >> 6)] = lnib[t];
    }

    // Everything issued so far completes here, in a wait the compiler sees
    // (otherwise its waits for the weights land inside the unit loop).
    wait_vmcnt<0>();
    __syncthreads();

    for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
        const int r = (int)(u / J), k0 = (int)(u - (int64_t)r * J) * kQ;
        const int np = min(kQ, N - k0);
        {   // stage C (columns past N read as zero) and the pair mask
            const int c = t >> 3, q = 4 * (t & 7);
            float4 a = cur.c0, b = cur.c1;
            if (q + 4 > np) {
                if (q + 0 >= np) a.x = b.x = 0.f;
                if (q + 1 >= np) a.y = b.y = 0.f;
                if (q + 2 >= np) a.z = b.z = 0.f;
                if (q + 3 >= np) a.w = b.w = 0.f;
            }
            *reinterpret_cast<float4*>(&cs[c * kCs + q]) = a;
            *reinterpret_cast<float4*>(&cs[(c + 64) * kCs + q]) = b;
            if (t < kQ) mq[t] = (t < np && (!mask || (cur.mr != 0 && cur.mk != 0))) ? 1.f : 0.f;
        }
        {   // LN_in of pair lp over d = 8 lq + i -> x hi / lo rows; dout -> dq
            const uint32_t zw[4] = {cur.zv.x, cur.zv.y, cur.zv.z, cur.zv.w};
            float x[8], s1 = 0.f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                x[2 * i] = __uint_as_float(zw[i] << 16);
                x[2 * i + 1] = __uint_as_float(zw[i] & 0xffff0000u);
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) s1 += x[i];
            const float mz = sum_lanes16(s1) * (1.f / kCz);
            float q2 = 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) { x[i] -= mz; q2 += x[i] * x[i]; }
            const float rz = rsqrtf(sum_lanes16(q2) * (1.f / kCz) + eps);
            uint32_t hw[4], lw[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int d = 8 * lq + 2 * i;
                const int dp = d + 4 * (d >> 6);             // padded position of d, d + 1
                const float x0 = x[2 * i] * rz * prm[2][dp] + prm[3][dp];
                const float x1 = x[2 * i + 1] * rz * prm[2][dp + 1] + prm[3][dp + 1];
                hw[i] = pack_bf16x2(x0, x1);
                lw[i] = pack_bf16x2(x0 - __uint_as_float(hw[i] << 16), x1 - __uint_as_float(hw[i] & 0xffff0000u));
            }
            *reinterpret_cast<uint4*>(act[2] + arow(lp, lq)) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
            *reinterpret_cast<uint4*>(act[3] + arow(lp, lq)) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
            float4 o0, o1;
            if constexpr (sizeof(TO) == 4) {
                o0 = cur.o.a;
                o1 = cur.o.b;
            } else {
                const uint4 v = cur.o.a;
                o0 = make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                                 __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
                o1 = make_float4(__uint_as_float(v.z << 16), __uint_as_float(v.z & 0xffff0000u),
                                 __uint_as_float(v.w << 16), __uint_as_float(v.w & 0xffff0000u));
            }
            *reinterpret_cast<float4*>(&dq[lp * kPq + 8 * lq]) = o0;
            *reinterpret_cast<float4*>(&dq[lp * kPq + 8 * lq + 4]) = o1;
        }
        load(u + gridDim.x, cur);                        // the next unit, into the released registers
        __syncthreads();
        float yh[8], rs;                                 // LN_out(C) normalised, c = lq + 16 i; 1 / std
        {   // LN_out of pair lp over c = lq + 16 i -> y hi / lo rows
            float s1 = 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) { yh[i] = cs[(lq + 16 * i) * kCs + lp]; s1 += yh[i]; }
            const float mu = sum_lanes16(s1) * (1.f / kCh);
            float q2 = 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) { yh[i] -= mu; q2 += yh[i] * yh[i]; }
            rs = rsqrtf(sum_lanes16(q2) * (1.f / kCh) + eps);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int c = lq + 16 * i;
                yh[i] *= rs;
                st_hilo(act[0], act[1], arow(lp, c >> 3) + 2 * (c & 7), yh[i] * prm[0][c] + prm[1][c]);
            }
        }
        __syncthreads();
        {   // u = y W_o^T, gg = x W_g^T (columns d = 16 w + col); du, dgg
            f32x4_t au[2], ag[2];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) au[mb] = ag[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int mb = 0; mb < 2; ++mb) {
                    const uint32_t o = arow(16 * mb + col, 4 * ks + kq);
                    au[mb] = mfma16(ld_frag(act[0], o), wo[ks], au[mb]);
                    ag[mb] = mfma16(ld_frag(act[2], o), wg[ks], ag[mb]);
                    au[mb] = mfma16(ld_frag(act[1], o), wo[ks], au[mb]);
                    ag[mb] = mfma16(ld_frag(act[3], o), wg[ks], ag[mb]);
                }
            // unit blocks of y and x (bf16 = the hi rows), channel-major
            *reinterpret_cast<uint4*>(b_y + u * (kCh * kQ) + sc * kQ + 8 * sq) = gather_col8(act[0], 8 * sq, sc);
            *reinterpret_cast<uint4*>(b_x + u * (kCh * kQ) + sc * kQ + 8 * sq) = gather_col8(act[2], 8 * sq, sc);
            const int d = 16 * w + col;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                float vu[4], vg[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int q = 16 * mb + 4 * kq + i;
                    const float o = dq[q * kPq + d] * mq[q];
                    const float g = sigmoidf_(ag[mb][i]);
                    vu[i] = o * g;
                    vg[i] = o * au[mb][i] * g * (1.f - g);
                    const uint32_t off = arow(q, d >> 3) + 2 * (d & 7);
                    st_hilo(act2[0], act2[1], off, vu[i]);
                    st_hilo(act2[2], act2[3], off, vg[i]);
                }
                const int64_t bo = u * (kCh * kQ) + d * kQ + 16 * mb + 4 * kq;
                *reinterpret_cast<uint2*>(b_du + bo) = pack4(vu[0], vu[1], vu[2], vu[3]);
                *reinterpret_cast<uint2*>(b_dgg + bo) = pack4(vg[0], vg[1], vg[2], vg[3]);
            }
        }
        __syncthreads();
        {   // dy = du W_o -> dq; dx_g = dgg W_g -> HBM (columns n = 16 w + col)
            f32x4_t ay[2], ax[2];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) ay[mb] = ax[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int mb = 0; mb < 2; ++mb) {
                    const uint32_t o = arow(16 * mb + col, 4 * ks + kq);
                    ay[mb] = mfma16(ld_frag(act2[0], o), wot[ks], ay[mb]);
                    ax[mb] = mfma16(ld_frag(act2[2], o), wgt[ks], ax[mb]);
                    ay[mb] = mfma16(ld_frag(act2[1], o), wot[ks], ay[mb]);
                    ax[mb] = mfma16(ld_frag(act2[3], o), wgt[ks], ax[mb]);
                }
            const int n = 16 * w + col;
            const auto rx = make_rsrc(dxg + ((int64_t)r * N + k0) * kCz, np * kCz * 4);   // pairs past N: dropped
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int q = 16 * mb + 4 * kq + i;
                    dq[q * kPq + n] = ay[mb][i];
                    bst_f32(rx, (q * kCz + n) * 4, ax[mb][i]);
                }
        }
        __syncthreads();
        {   // LN_out backward of pair lp: dC = rs (dy gamma - mean(dy gamma) - yh mean(dy gamma yh))
            float dy[8], s1 = 0.f, s2 = 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int c = lq + 16 * i;
                dy[i] = dq[lp * kPq + c];
                const float dh = dy[i] * prm[0][c];
                s1 += dh;
                s2 += dh * yh[i];
            }
            s1 = sum_lanes16(s1) * (1.f / kCh);
            s2 = sum_lanes16(s2) * (1.f / kCh);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int c = lq + 16 * i;
                dct[c * kCs + lp] = rs * (dy[i] * prm[0][c] - s1 - yh[i] * s2);
                accg[i] += dy[i] * yh[i];
                accb[i] += dy[i];
            }
        }
        __syncthreads();
        {   // dC row r, columns k0 + 8 sq .. + 7 of channel sc into the panel
            const float4 a = *reinterpret_cast<const float4*>(&dct[sc * kCs + 8 * sq]);
            const float4 b = *reinterpret_cast<const float4*>(&dct[sc * kCs + 8 * sq + 4]);
            *reinterpret_cast<uint4*>(dCp + panel_off(pg, sc, r, k0 + 8 * sq)) =
                make_uint4(pack_bf16x2(a.x, a.y), pack_bf16x2(a.z, a.w), pack_bf16x2(b.x, b.y), pack_bf16x2(b.z, b.w));
        }
    }
    // per-work-group sums over the pairs lanes (lp) through LDS
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        cs[lp * kCh + lq + 16 * i] = accg[i];
        dct[lp * kCh + lq + 16 * i] = accb[i];
    }
    __syncthreads();
    if (t < 2 * kCh) {
        const float* src = t < kCh ? cs : dct;
        const int c = t & (kCh - 1);
        float s = 0.f;
        for (int q = 0; q < kQ; ++q) s += src[q * kCh + c];
        partial[((int64_t)blockIdx.x * 2 + (t >> 7)) * kCh + c] = s;
    }
}

// Projection backward.  Unit (r, kb) of dA / dB; its pairs are P(q) = (r, k)
// (outgoing) or (k, r) (incoming).  Recompute x = LN_in(z) and the four
// projections p_a, g_a, p_b, g_b (pre-sigmoid gates); then
//   dpa = da m s_a,  dga = da m p_a s_a (1 - s_a)  (the same for b),
//   dx = dx_g + [dpa dga dpb dgb] [W_a; W_ga; W_b; W_gb],  dz = LN_in backward of dx
// (the four gradients enter that product rounded to bf16; x enters the
// projections as bf16 hi + lo).
// Writes dz, unit blocks dpa, dga, dpb, dgb, x, and per-work-group sums of
// dgamma_in, dbeta_in at partial[(2 wg + {0, 1}) * 128 + d].
//
// Wave w owns 32 output columns of both products and keeps both weight
// slices in registers: rows 32 w + col of W_a, W_ga, W_b, W_gb for the
// projections and row d = 32 w + col of [W_a^T | W_ga^T | W_b^T | W_gb^T]
// (512 long) for dx, 256 registers; so the kernel runs 4 waves, one per
// SIMD, each with the whole register file.  Products on
// v_mfma_f32_32x32x16_bf16: lane l supplies row (column) l % 32 and k values
// 8 (l / 32) .. + 7; the result gives lane l column l % 32 and rows
// 8 (i / 4) + 4 (l / 32) + i % 4, i = 0 .. 15.
constexpr int kPT = 256;      // threads of the projection backward
constexpr int kPq4 = 136;     // [pair][channel] row stride: rows 4 apart land 32 banks apart
// Padded bf16 row tiles: a row of 128 (x) or 512 (the four gradients)
// values plus one 16-byte chunk, so the 16 rows an operand read touches
// start 4 banks apart (conflict-free) and every access is the lane's base
// address plus an immediate offset.
constexpr int kXrow = 256 + 16;
constexpr int kGrow = 1024 + 16;

// 8 bf16 of column `col` of a padded [q][128] bf16 tile, rows q0 .. q0 + 7, packed.
__device__ __forceinline__ uint4 gather_col8p(const char* tile, int q0, int col) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t a = *reinterpret_cast<const bf16_t*>(tile + (q0 + 2 * i) * kXrow + 2 * col);
        const uint32_t b = *reinterpret_cast<const bf16_t*>(tile + (q0 + 2 * i + 1) * kXrow + 2 * col);
        w[i] = a | (b << 16);
    }
    return make_uint4(w[0], w[1], w[2], w[3]);
}

template <bool INCOMING>
__global__ __attribute__((amdgpu_flat_work_group_size(kPT, kPT), amdgpu_waves_per_eu(1, 1)))
void k_projection_backward(
    const bf16_t* __restrict__ z, const uint8_t* __restrict__ mask, int N, int64_t units, const float* __restrict__ dA,
    const float* __restrict__ dB, const float* __restrict__ dxg, const bf16_t* __restrict__ wproj,
    const bf16_t* __restrict__ wprojt, const float* __restrict__ lniw, const float* __restrict__ lnib, float eps,
    bf16_t* __restrict__ dz, bf16_t* __restrict__ b_dpa, bf16_t* __restrict__ b_dga, bf16_t* __restrict__ b_dpb,
    bf16_t* __restrict__ b_dgb, bf16_t* __restrict__ b_x, float* __restrict__ partial) {
    __shared__ __align__(16) float das[kCh * kCs];       // da [c][q]
    __shared__ __align__(16) float dbs[kCh * kCs];       // db [c][q]
    __shared__ __align__(16) char xa[2][kQ * kXrow];     // x hi, x lo  [q][128]
    __shared__ __align__(16) char d4[kQ * kGrow];        // bf16 [q][dpa | dga | dpb | dgb]
    __shared__ __align__(16) float dxs[kQ * kPq4];       // dx from the projections [q][d]
    __shared__ __align__(16) float xhs[kQ * kPq4];       // LN_in(z) normalised [q][d]
    __shared__ float rzs[kQ];                            // 1 / std of LN_in per pair
    __shared__ float prm[2][128];                        // gamma_in, beta_in
    __shared__ float mq[kQ];
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int lp = t >> 3, lq = t & 7;                   // LayerNorm: pair lp, d = 16 lq .. + 15
    const int J = (N + kQ - 1) / kQ;
    auto pair_of = [&](int r, int k) -> int64_t { return INCOMING ? (int64_t)k * N + r : (int64_t)r * N + k; };


    // One unit's loads, issued one unit ahead; dx_g is fetched separately
    // (it is used last).  Nothing here reads the loaded registers.
    struct Pre {
        float4 a[4], b[4];       // dA, dB block floats 4 (t + 256 s) ..
        uint4 z0, z1;            // z of pair lp, channels 16 lq .. + 15
        uint32_t mr, mk;
    };
    // Byte distance between consecutive pairs of a unit in [pair][c_z]
    // tensors: adjacent columns (outgoing) or adjacent rows (incoming).
    const uint32_t step2 = INCOMING ? (uint32_t)N * kCz * 2 : kCz * 2;   // bf16
    const uint32_t step4 = 2 * step2;                                    // fp32
    auto load = [&](int64_t u, Pre& p) {
        const bool valid = u < units;                     // past the end: zero-size resources
        const int64_t uu = valid ? u : 0;
        const int r = (int)(uu / J), k0 = (int)(uu - (int64_t)r * J) * kQ;
        const int np = min(kQ, N - k0);
        const auto ra = make_rsrc(dA + uu * (kCh * kQ), valid ? kCh * kQ * 4 : 0);
        const auto rb = make_rsrc(dB + uu * (kCh * kQ), valid ? kCh * kQ * 4 : 0);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            p.a[s] = bld_f4(ra, 16 * (t + kPT * s));
            p.b[s] = bld_f4(rb, 16 * (t + kPT * s));
        }
        const auto rzr = make_rsrc(z + pair_of(r, k0) * kCz, valid ? (np - 1) * step2 + kCz * 2 : 0);
        p.z0 = buf_load16(rzr, lp * step2 + 32 * lq);
        p.z1 = buf_load16(rzr, lp * step2 + 32 * lq + 16);
        const auto rm = make_rsrc(mask, (valid && mask) ? (uint32_t)N : 0u);
        p.mr = bld_u8(rm, opaque(r));                    // per lane: a uniform load would be waited for at once
        p.mk = bld_u8(rm, k0 + (t & (kQ - 1)));
    };
    auto load_dxg = [&](int64_t u, float4 (&g)[4]) {
        const bool valid = u < units;
        const int64_t uu = valid ? u : 0;
        const int r = (int)(uu / J), k0 = (int)(uu - (int64_t)r * J) * kQ;
        const int np = min(kQ, N - k0);
        const auto rg = make_rsrc(dxg + pair_of(r, k0) * kCz, valid ? (np - 1) * step4 + kCz * 4 : 0);
#pragma unroll
        for (int s = 0; s < 4; ++s) g[s] = bld_f4(rg, lp * step4 + 64 * lq + 16 * s);
    };

    float accg[16], accb[16];                            // dgamma_in, dbeta_in of d = 16 lq + i
#pragma unroll
    for (int i = 0; i < 16; ++i) accg[i] = accb[i] = 0.f;
    Pre cur;
    float4 xg[4];
    load(blockIdx.x, cur);
    load_dxg(blockIdx.x, xg);
    bf16x8_t wp[32], wt[32];   // wp[8 m + ks]: map m, k = 16 ks + 8 hi;  wt[ks]: k = 16 ks + 8 hi
    {
        const int col = lane & 31, hi = lane >> 5;
#pragma unroll
        for (int j = 0; j < 32; ++j) {
            wp[j] = *reinterpret_cast<const bf16x8_t*>(
                wproj + ((int64_t)w * 128 + (j >> 3) * 32 + col) * 128 + 16 * (j & 7) + 8 * hi);
            wt[j] = *reinterpret_cast<const bf16x8_t*>(wprojt + (int64_t)(32 * w + col) * 512 + 16 * j + 8 * hi);
        }
    }
    if (t < 128) {
        prm[0][t] = lniw[t];
        prm[1][t] = lnib[t];
    }
    // Everything issued so far completes here, in a wait the compiler sees:
    // otherwise it places the waits for the weights inside the unit loop,
    // where on later passes they stall on the next unit's prefetch.
    wait_vmcnt<0>();
    __syncthreads();   // the first unit's LN_in reads prm before the loop's first barrier

    for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
        const int r = (int)(u / J), k0 = (int)(u - (int64_t)r * J) * kQ;
        const int np = min(kQ, N - k0);
        float xh[16], rz;   // LN_in(z) normalised, d = 16 lq + i, and 1 / std: to LDS after the barrier
        {   // stage da, db and the mask; LN_in of pair lp -> x hi / lo rows
            const int t = opaque(threadIdx.x), lp = t >> 3, lq = t & 7;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int c = (t >> 3) + 32 * s, q = 4 * (t & 7);
                *reinterpret_cast<float4*>(&das[c * kCs + q]) = cur.a[s];
                *reinterpret_cast<float4*>(&dbs[c * kCs + q]) = cur.b[s];
            }
            if (t < kQ) mq[t] = (t < np && (!mask || (cur.mr != 0 && cur.mk != 0))) ? 1.f : 0.f;
            const uint32_t zw[8] = {cur.z0.x, cur.z0.y, cur.z0.z, cur.z0.w, cur.z1.x, cur.z1.y, cur.z1.z, cur.z1.w};
            float s1 = 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                xh[2 * i] = __uint_as_float(zw[i] << 16);
                xh[2 * i + 1] = __uint_as_float(zw[i] & 0xffff0000u);
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) s1 += xh[i];
            const float mz = sum_lanes8(s1) * (1.f / kCz);
            float q2 = 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) { xh[i] -= mz; q2 += xh[i] * xh[i]; }
            rz = rsqrtf(sum_lanes8(q2) * (1.f / kCz) + eps);
            uint32_t hw[8], lw[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int d = 16 * lq + 2 * i;
                xh[2 * i] *= rz;
                xh[2 * i + 1] *= rz;
                const float x0 = xh[2 * i] * prm[0][d] + prm[1][d];
                const float x1 = xh[2 * i + 1] * prm[0][d + 1] + prm[1][d + 1];
                hw[i] = pack_bf16x2(x0, x1);
                lw[i] = pack_bf16x2(x0 - __uint_as_float(hw[i] << 16), x1 - __uint_as_float(hw[i] & 0xffff0000u));
            }
            *reinterpret_cast<uint4*>(xa[0] + lp * kXrow + 32 * lq) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
            *reinterpret_cast<uint4*>(xa[0] + lp * kXrow + 32 * lq + 16) = make_uint4(hw[4], hw[5], hw[6], hw[7]);
            *reinterpret_cast<uint4*>(xa[1] + lp * kXrow + 32 * lq) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
            *reinterpret_cast<uint4*>(xa[1] + lp * kXrow + 32 * lq + 16) = make_uint4(lw[4], lw[5], lw[6], lw[7]);
        }
        load(u + gridDim.x, cur);                        // next unit's dA, dB, z, mask
        __syncthreads();
        {   // xhs and rzs are read by the previous unit's last phase: written only past the barrier
            const int t = opaque(threadIdx.x), lp = t >> 3, lq = t & 7;
#pragma unroll
            for (int s = 0; s < 4; ++s)
                *reinterpret_cast<float4*>(&xhs[lp * kPq4 + 16 * lq + 4 * s]) =
                    make_float4(xh[4 * s], xh[4 * s + 1], xh[4 * s + 2], xh[4 * s + 3]);
            if (lq == 0) rzs[lp] = rz;
        }
        {   // projections of channels c = 32 w + col; the four gradients
            const int lo = opaque(lane), col = lo & 31, hi = lo >> 5;
            const int c = 32 * w + col;
#pragma unroll
            for (int h = 0; h < 2; ++h) {                // h = 0: (p_a, g_a), h = 1: (p_b, g_b)
                f32x16_t ap, ag;
#pragma unroll
                for (int i = 0; i < 16; ++i) ap[i] = ag[i] = 0.f;
#pragma unroll
                for (int ks = 0; ks < 8; ++ks) {
                    const uint32_t o = col * kXrow + 32 * ks + 16 * hi;
                    const bf16x8_t xhi = ld_frag(xa[0], o), xlo = ld_frag(xa[1], o);
                    ap = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xhi, wp[16 * h + ks], ap, 0, 0, 0);
                    ag = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xhi, wp[16 * h + 8 + ks], ag, 0, 0, 0);
                    ap = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xlo, wp[16 * h + ks], ap, 0, 0, 0);
                    ag = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xlo, wp[16 * h + 8 + ks], ag, 0, 0, 0);
                }
                const float* dsrc = h ? dbs : das;
                bf16_t* bp = h ? b_dpb : b_dpa;
                bf16_t* bg = h ? b_dgb : b_dga;
                const int kp = 256 * h + c, kg = 256 * h + 128 + c;
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    const int q0 = 8 * a + 4 * hi;
                    const float4 dd4 = *reinterpret_cast<const float4*>(&dsrc[c * kCs + q0]);
                    const float dd[4] = {dd4.x, dd4.y, dd4.z, dd4.w};
                    float vp[4], vg[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int q = q0 + i;
                        const bool m = mq[q] != 0.f;
                        const float s = sigmoidf_(ag[4 * a + i]);
                        vp[i] = m ? dd[i] * s : 0.f;
                        vg[i] = m ? dd[i] * ap[4 * a + i] * s * (1.f - s) : 0.f;
                        *reinterpret_cast<bf16_t*>(d4 + q * kGrow + 2 * kp) = f2bf(vp[i]);
                        *reinterpret_cast<bf16_t*>(d4 + q * kGrow + 2 * kg) = f2bf(vg[i]);
                    }
                    const int64_t bo = u * (kCh * kQ) + c * kQ + q0;
                    *reinterpret_cast<uint2*>(bp + bo) = pack4(vp[0], vp[1], vp[2], vp[3]);
                    *reinterpret_cast<uint2*>(bg + bo) = pack4(vg[0], vg[1], vg[2], vg[3]);
                }
            }
        }
        __syncthreads();
        {   // dx (projection part) of columns d = 32 w + col over K = 512; unit block of x
            const int lo = opaque(lane), col = lo & 31, hi = lo >> 5;
            f32x16_t ax;
#pragma unroll
            for (int i = 0; i < 16; ++i) ax[i] = 0.f;
#pragma unroll
            for (int ks = 0; ks < 32; ++ks)
                ax = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ld_frag(d4, col * kGrow + 32 * ks + 16 * hi), wt[ks], ax, 0, 0, 0);
            const int to = opaque(threadIdx.x), sc = to >> 1, sh = to & 1;
            bf16_t* xb = b_x + u * (kCh * kQ) + sc * kQ + 16 * sh;
            reinterpret_cast<uint4*>(xb)[0] = gather_col8p(xa[0], 16 * sh, sc);
            reinterpret_cast<uint4*>(xb)[1] = gather_col8p(xa[0], 16 * sh + 8, sc);
            const int d = 32 * w + col;
#pragma unroll
            for (int i = 0; i < 16; ++i) dxs[(8 * (i >> 2) + 4 * hi + (i & 3)) * kPq4 + d] = ax[i];
        }
        __syncthreads();
        {   // LN_in backward of pair lp: dz = rz (dx gamma - mean(dx gamma) - xh mean(dx gamma xh))
            const int t = opaque(threadIdx.x), lp = t >> 3, lq = t & 7;
            float dx[16], xh[16], s1 = 0.f, s2 = 0.f;
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const float4 p = *reinterpret_cast<const float4*>(&dxs[lp * kPq4 + 16 * lq + 4 * s]);
                const float4 hh = *reinterpret_cast<const float4*>(&xhs[lp * kPq4 + 16 * lq + 4 * s]);
                dx[4 * s] = p.x + xg[s].x;
                dx[4 * s + 1] = p.y + xg[s].y;
                dx[4 * s + 2] = p.z + xg[s].z;
                dx[4 * s + 3] = p.w + xg[s].w;
                xh[4 * s] = hh.x;
                xh[4 * s + 1] = hh.y;
                xh[4 * s + 2] = hh.z;
                xh[4 * s + 3] = hh.w;
            }
            const float rz = rzs[lp];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float dh = dx[i] * prm[0][16 * lq + i];
                s1 += dh;
                s2 += dh * xh[i];
                accg[i] += dx[i] * xh[i];
                accb[i] += dx[i];
            }
            s1 = sum_lanes8(s1) * (1.f / kCz);
            s2 = sum_lanes8(s2) * (1.f / kCz);
            uint32_t o[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int d = 16 * lq + 2 * i;
                o[i] = pack_bf16x2(rz * (dx[2 * i] * prm[0][d] - s1 - xh[2 * i] * s2),
                                   rz * (dx[2 * i + 1] * prm[0][d + 1] - s1 - xh[2 * i + 1] * s2));
            }
            const auto rd = make_rsrc(dz + pair_of(r, k0) * kCz, (np - 1) * step2 + kCz * 2);   // pairs past N: dropped
            bst_u4(rd, lp * step2 + 32 * lq, make_uint4(o[0], o[1], o[2], o[3]));
            bst_u4(rd, lp * step2 + 32 * lq + 16, make_uint4(o[4], o[5], o[6], o[7]));
        }
        load_dxg(u + gridDim.x, xg);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        das[lp * kCz + 16 * lq + i] = accg[i];
        dbs[lp * kCz + 16 * lq + i] = accb[i];
    }
    __syncthreads();
    {
        const float* src = t < kCz ? das : dbs;
        const int d = t & (kCz - 1);
        float s = 0.f;
        for (int q = 0; q < kQ; ++q) s += src[q * kCz + d];
        partial[((int64_t)blockIdx.x * 2 + (t >> 7)) * kCz + d] = s;
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
// Four weight gradients that share their second operand (W_a, W_ga, W_b,
// W_gb all multiply the x blocks): sum over units of U_o V^T for o = 0..3,
// reading each unit's V block once instead of four times.  8 waves: wave w
// owns rows 32 (w % 4) .. + 31 of outputs 2 (w / 4) and 2 (w / 4) + 1
// (two 32 x 128 accumulators); the next unit's operands are loaded while
// the current one is multiplied.  Partials: [o][grid][128][128].
struct Wgrad4Args {
    const bf16_t* u[4];
};

__global__ __launch_bounds__(512) void k_wgrad4(Wgrad4Args a, const bf16_t* __restrict__ V, int64_t units,
                                                float* __restrict__ partial) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int rl = lane & 31, hi = lane >> 5;
    const int rb = 32 * (w & 3), o0 = 2 * (w >> 2);
    const bf16_t* U0 = a.u[o0];
    const bf16_t* U1 = a.u[o0 + 1];
    f32x16_t acc[2][4];
#pragma unroll
    for (int o = 0; o < 2; ++o)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[o][j][r] = 0.f;
    struct Ops { bf16x8_t a[2][2], b[4][2]; };
    auto load = [&](int64_t u, Ops& p) {
        const int64_t uu = u < units ? u : units - 1;   // past the end: a repeat, never multiplied
        const int64_t base = uu * (kCh * kQ);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const int64_t ra = base + (rb + rl) * kQ + 16 * ks + 8 * hi;
            p.a[0][ks] = *reinterpret_cast<const bf16x8_t*>(U0 + ra);
            p.a[1][ks] = *reinterpret_cast<const bf16x8_t*>(U1 + ra);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                p.b[j][ks] = *reinterpret_cast<const bf16x8_t*>(V + base + (32 * j + rl) * kQ + 16 * ks + 8 * hi);
        }
    };
    Ops cur, nxt;
    load(blockIdx.x, cur);
    for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
        load(u + gridDim.x, nxt);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int o = 0; o < 2; ++o)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[o][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cur.a[o][ks], cur.b[j][ks], acc[o][j], 0, 0, 0);
        cur = nxt;
    }
    // lane holds column 32 j + rl; register r holds row rb + 8 (r / 4) + 4 hi + r % 4
#pragma unroll
    for (int o = 0; o < 2; ++o) {
        float* pw = partial + ((int64_t)(o0 + o) * gridDim.x + blockIdx.x) * (kCh * kCh);
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) pw[(rb + 8 * (r >> 2) + 4 * hi + (r & 3)) * kCh + 32 * j + rl] = acc[o][j][r];
    }
}

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
    const int64_t units = (N + 1) / 2 * ((N + kResJ - 1) / kResJ);   // row pairs x column blocks
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

int backward_grid(int64_t units, int cus, int per_cu) {
    return (int)(units < (int64_t)per_cu * cus ? units : (int64_t)per_cu * cus);
}

hipError_t launch_epilogue_backward(int out_dtype, const DeviceWeights& w, const float* C, const void* z,
                                    const uint8_t* mask, const void* dout, int64_t N, void* dCp, float* dxg,
                                    const BackwardBlocks& bb, float* partial, int grid, hipStream_t s) {
    const int64_t units = N * ((N + 31) / 32);
    if (out_dtype == 0)
        hipLaunchKernelGGL(k_epilogue_backward<float>, dim3(grid), dim3(kBT), 0, s, C, (const bf16_t*)z, mask,
                           (const float*)dout, (int)N, units, w.epi_bf, w.epit_bf, w.ln_in_w, w.ln_in_b, w.ln_out_w,
                           w.ln_out_b, w.eps, (bf16_t*)dCp, dxg, bb.du, bb.y, bb.dgg, bb.xe, partial);
    else
        hipLaunchKernelGGL(k_epilogue_backward<bf16_t>, dim3(grid), dim3(kBT), 0, s, C, (const bf16_t*)z, mask,
                           (const bf16_t*)dout, (int)N, units, w.epi_bf, w.epit_bf, w.ln_in_w, w.ln_in_b,
                           w.ln_out_w, w.ln_out_b, w.eps, (bf16_t*)dCp, dxg, bb.du, bb.y, bb.dgg, bb.xe, partial);
    return hipGetLastError();
}

hipError_t launch_projection_backward(const DeviceWeights& w, const void* z, const uint8_t* mask, int64_t N,
                                      int incoming, const float* dA, const float* dB, const float* dxg, void* dz,
                                      const BackwardBlocks& bb, float* partial, int grid, hipStream_t s) {
    const int64_t units = N * ((N + 31) / 32);
    if (incoming)
        hipLaunchKernelGGL(k_projection_backward<true>, dim3(grid), dim3(kPT), 0, s, (const bf16_t*)z, mask, (int)N,
                           units, dA, dB, dxg, w.proj_bf, w.projt_bf, w.ln_in_w, w.ln_in_b, w.eps, (bf16_t*)dz,
                           bb.dpa, bb.dga, bb.dpb, bb.dgb, bb.xp, partial);
    else
        hipLaunchKernelGGL(k_projection_backward<false>, dim3(grid), dim3(kPT), 0, s, (const bf16_t*)z, mask, (int)N,
                           units, dA, dB, dxg, w.proj_bf, w.projt_bf, w.ln_in_w, w.ln_in_b, w.eps, (bf16_t*)dz,
                           bb.dpa, bb.dga, bb.dpb, bb.dgb, bb.xp, partial);
    return hipGetLastError();
}

hipError_t launch_wgrad(const bf16_t* U, const bf16_t* V, int64_t N, float* partial, int grid, hipStream_t s) {
    const int64_t units = N * ((N + 31) / 32);
    hipLaunchKernelGGL(k_wgrad, dim3(grid), dim3(256), 0, s, U, V, units, partial);
    return hipGetLastError();
}

hipError_t launch_wgrad4(const bf16_t* const U[4], const bf16_t* V, int64_t N, float* partial, int grid,
                         hipStream_t s) {
    const int64_t units = N * ((N + 31) / 32);
    Wgrad4Args a{{U[0], U[1], U[2], U[3]}};
    hipLaunchKernelGGL(k_wgrad4, dim3(grid), dim3(512), 0, s, a, V, units, partial);
    return hipGetLastError();
}

hipError_t launch_sum_parts(const float* in, int parts, int64_t stride, int n, float* out, hipStream_t s) {
    hipLaunchKernelGGL(k_sum_parts, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, in, parts, stride, n, out);
    return hipGetLastError();
}

}  // namespace trimul
