// K1: input LayerNorm + gated a/b projections + pair mask, writing the
// channel-major operands of the contraction (Section 3.3: a, b are gated
// projections of z; Eq. 2 / Eq. 3 pick which token index is contracted).
//
// Work unit: a "line" of 64 pairs that share one output row.  Outgoing line
// (r, k0): pairs (r, k0..k0+63), A[c][r][k0+p] = a(r, k0+p).  Incoming line
// (r, k0): pairs (k0..k0+63, r), A[c][r][k0+p] = a(k0+p, r).  Either way the
// 64 results of one channel are contiguous in A and B.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace trimul {
namespace {

constexpr int kLine = 64;   // pairs per work unit

// Scalar (VALU) fp32 version; it serves the fp32 storage path.
template <typename T, bool INCOMING>
__global__ __launch_bounds__(256) void k1_project_valu(
    const T* __restrict__ z, const uint8_t* __restrict__ mask, int64_t N, int64_t nchunk,
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
            const int64_t off = panel_off(panel_geom(N, N), c, r, k0 + p);
            Store<T>::st(A + off, a);
            Store<T>::st(B + off, b);
        }
    }
}


// ------------------------------------------------------------ bf16 MFMA
//
// Persistent kernel, 4 waves, work unit = line of 32 pairs.  Wave g owns
// hidden channels [32 g, 32 g + 32): its 128 weight rows (W_a, W_ga, W_b,
// W_gb of those channels) stay in VGPRs for the whole kernel as the MFMA A
// operand, so the 4 x 32 outputs of a channel land in the same lane and
// register and the gating is element-wise in registers.
//
// z and the token mask reach LDS through a 3-stage ring filled by
// direct-to-LDS buffer loads two lines ahead of the line being computed, so
// the HBM latency of z hides behind two lines of work.  Every wave issues
// the same number of vector-memory instructions per line (3 loads, 4 stores,
// tails included), which makes the vmcnt waits exact constants.
//
// Precision: the matrix cores take fp16 operands, 11 significant bits
// against bf16's 8.  The weights (bf16 values) and the LayerNormed x
// (fp32) are scaled by powers of two chosen at initialisation so that the
// largest possible operand lies in [2^14, 2^15]: the weights convert
// exactly (down to 2^-17 of that largest entry) and x rounds once to
// 2^-11 relative, with no overflow and no subnormal x.  So values and gates
// carry ~11 bits, and the main error of a and b stays their bf16 store.
// The gating undoes the scales (DeviceWeights::K1Scales) inside the
// logistic at no extra instruction.
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
constexpr int kP1 = 32;                 // pairs per line
constexpr int kXRow = kCz * 2;          // bytes of one bf16 row of 128 channels (256)
constexpr int kZSt = kP1 * kXRow;       // z bytes of one line (8 KB)
constexpr int kMSt = 4 * 256;           // per-wave token-mask bytes of one line
constexpr int kSt = kZSt + kMSt;        // one ring stage
constexpr int kRing = 3;

// x rows [p][128] bf16: 16-byte chunk q of row p lives at slot q ^ (p & 15).
__device__ __forceinline__ uint32_t xoff(int p, int chunk) {
    return (uint32_t)(p * kXRow + ((chunk ^ (p & 15)) << 4));
}

// The operands are M x K: operand row i (M of them) and contraction index k
// (K).  Outgoing, pair (i, k) is z[i][k]; incoming, pair (k, i) is z[k][i];
// z rows are ldz pairs apart (the full update: M = K = ldz = N; a device
// tile: its rows and columns).  tmask: the staged 0/1 token bytes, the
// k-range's at [0, ceil(K/32)*32) (zero past K) and operand row i's at
// rmoff + i; mrange bytes of it are readable.
template <bool INCOMING>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(2, 2)))
void k1_project_mfma(const bf16_t* __restrict__ z, int ldz, const uint8_t* __restrict__ tmask, int rmoff,
                     int mrange, int M, int K, int nlines, const uint16_t* __restrict__ wproj,
                     const float* __restrict__ lnw, const float* __restrict__ lnb, float eps,
                     DeviceWeights::K1Scales ks, bf16_t* __restrict__ A, bf16_t* __restrict__ B) {
    __shared__ __attribute__((aligned(16))) char ring[kRing * kSt];     // z rows [p][256 B], mask
    __shared__ __attribute__((aligned(16))) char xs[kP1 * kXRow];      // x (fp16, scaled)
    __shared__ __attribute__((aligned(16))) float os[2][kCh][kP1];      // a, b as [c][p]
    // LayerNorm gain, bias; channel c at (c / 16) * 20 + c % 16, so that the
    // 8 broadcast addresses of a read (c = 16 lq + 4 i) fall in distinct banks
    __shared__ __attribute__((aligned(16))) float gb[2][8 * 20];
    const int t = threadIdx.x, lane = t & 63;
    const int g = __builtin_amdgcn_readfirstlane(t >> 6);
    const int lp = t >> 3, lq = t & 7;     // LayerNorm: pair lp, channels 16 lq .. 16 lq + 15
    // Line order: rows fastest (line = kc * M + r covers pairs k0 = 32 kc ..
    // k0 + 31 of operand row r), and the work-groups of one XCD take consecutive
    // lines; the grid's lines of one round then fill whole 256-row blocks of
    // the operands and read long runs of z in either direction.
    const int G = gridDim.x;
    const int first = (G & 7) == 0 ? (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3) : blockIdx.x;

    // Ring fill.  Stage row p holds pair k0 + p of the line; its 16-byte
    // chunk q sits at slot q ^ (p & 1), so that the LayerNorm reads of two
    // neighbouring rows hit disjoint banks.  Wave g loads rows 8 g .. 8 g + 7
    // (two 1 KB loads: lane i -> row 8 g + 4 h + i / 16, slot i % 16) and its
    // own copy of the line's mask bytes: m[k0 .. k0 + 31] at 0, the dword of
    // row r's byte at 32.  Lines past the end load nothing (zero-size
    // descriptor).
    const uint32_t zstep = INCOMING ? (uint32_t)ldz * kXRow : (uint32_t)kXRow;   // bytes between pairs
    const uint32_t ring_base = lds_addr(ring);
    const int drow = g * 8 + (lane >> 4);
    const uint32_t dchunk = (uint32_t)(((lane & 15) ^ (drow & 1)) << 4);
    const uint32_t dv0 = (uint32_t)drow * zstep + dchunk, dv1 = (uint32_t)(drow + 4) * zstep + dchunk;
    auto issue = [&](int line, int stage) {
        const bool valid = line < nlines;
        int r = 0, k0 = 0;
        if (valid) {
            const int kc = line / M;
            r = line - kc * M;
            k0 = kc * kP1;
        }
        const int np = valid ? min(kP1, K - k0) : 0;
        const int64_t pair0 = INCOMING ? (int64_t)k0 * ldz + r : (int64_t)r * ldz + k0;
        const v4i_t rz = buffer_desc(z + pair0 * kCz, np > 0 ? (uint32_t)(np - 1) * zstep + kXRow : 0u);
        const uint32_t st = ring_base + (uint32_t)(stage * kSt);
        lds_load16(rz, dv0, 0, st + g * 2048);
        lds_load16(rz, dv1, 0, st + g * 2048 + 1024);
        const v4i_t rm = buffer_desc(tmask, valid ? (uint32_t)mrange : 0u);
        const uint32_t mo = lane < 8 ? (uint32_t)(k0 + 4 * lane) : lane == 8 ? (uint32_t)(rmoff + (r & ~3)) : 0xfffffff0u;
        lds_load4(rm, mo, 0, st + kZSt + g * 256);
    };
    issue(first, 0);
    issue(first + G, 1);

    f16x8_t w[4][8];
#pragma unroll
    for (int ob = 0; ob < 4; ++ob)
#pragma unroll
        for (int kq = 0; kq < 8; ++kq)
            w[ob][kq] = *reinterpret_cast<const f16x8_t*>(
                wproj + (size_t)(g * 128 + ob * 32 + (lane & 31)) * kCz + kq * 16 + 8 * (lane >> 5));
    if (t < kCz) {
        gb[0][(t >> 4) * 20 + (t & 15)] = lnw[t];
        gb[1][(t >> 4) * 20 + (t & 15)] = lnb[t];
    }
    const PanelGeom pg = panel_geom(M, K);
    // Store mapping: thread t writes pairs 8 (t & 3) .. 8 (t & 3) + 7 of
    // channel (t >> 2) + 64 (i & 1) of A (i < 2) or B (i >= 2).
    const int64_t ch_stride = panel_elems(pg);
    const int64_t st_lane = (t >> 2) * ch_stride + 8 * (t & 3);

    int stage = 0;
    for (int it = 0, line = first; line < nlines; ++it, line += G) {
        // Vector-memory instructions issued after this line's loads: the
        // next line's loads (3) and, from the second line on, the 4 stores
        // of every line in between.
        if (it == 0) wait_vmcnt_pinned<3>();
        else if (it == 1) wait_vmcnt_pinned<3 + 4>();
        else wait_vmcnt_pinned<3 + 4 + 4>();
        __syncthreads();
        issue(line + 2 * G, stage == 0 ? 2 : stage - 1);   // into the stage read one line ago
        const char* zs = ring + stage * kSt;
        stage = stage == 2 ? 0 : stage + 1;

        // LayerNorm of pair lp over 128 channels (8 lanes x 16 channels).
        float v[16];
        {
            const uint4 z0 = *reinterpret_cast<const uint4*>(zs + lp * kXRow + (((2 * lq) ^ (lp & 1)) << 4));
            const uint4 z1 = *reinterpret_cast<const uint4*>(zs + lp * kXRow + (((2 * lq + 1) ^ (lp & 1)) << 4));
            const uint32_t u[8] = {z0.x, z0.y, z0.z, z0.w, z1.x, z1.y, z1.z, z1.w};
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                v[2 * i] = __uint_as_float(u[i] << 16);
                v[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
            }
        }
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) s += v[i];
        s = sum_lanes8(s);
        const float mu = s * (1.0f / kCz);
        float q2 = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            v[i] -= mu;
            q2 += v[i] * v[i];
        }
        q2 = sum_lanes8(q2);
        const float rs = rsqrtf(q2 * (1.0f / kCz) + eps);
        float gam[16], bet[16];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float4 a4 = *reinterpret_cast<const float4*>(&gb[0][20 * lq + 4 * i]);
            const float4 b4 = *reinterpret_cast<const float4*>(&gb[1][20 * lq + 4 * i]);
            gam[4 * i] = a4.x; gam[4 * i + 1] = a4.y; gam[4 * i + 2] = a4.z; gam[4 * i + 3] = a4.w;
            bet[4 * i] = b4.x; bet[4 * i + 1] = b4.y; bet[4 * i + 2] = b4.z; bet[4 * i + 3] = b4.w;
        }
        f16x8_t xh[2];
#pragma unroll
        for (int i = 0; i < 16; ++i) xh[i >> 3][i & 7] = (_Float16)(v[i] * rs * gam[i] + bet[i]);
        // A masked pair (and a ragged line's tail: the staged mask is zero
        // past K) gets x = 0, so W x and with it a and b are exactly 0; the
        // AND also clears what a NaN in z would have left.
        const int kc = line / M, r0 = line - kc * M, k0 = kc * kP1;
        const uint8_t* ms = reinterpret_cast<const uint8_t*>(zs + kZSt + g * 256);   // this wave's copy
        const uint32_t keep = (ms[lp] & ms[32 + (r0 & 3)]) ? 0xffffffffu : 0u;
        uint4 x0 = __builtin_bit_cast(uint4, xh[0]), x1 = __builtin_bit_cast(uint4, xh[1]);
        x0 = make_uint4(x0.x & keep, x0.y & keep, x0.z & keep, x0.w & keep);
        x1 = make_uint4(x1.x & keep, x1.y & keep, x1.z & keep, x1.w & keep);
        *reinterpret_cast<uint4*>(xs + xoff(lp, 2 * lq)) = x0;
        *reinterpret_cast<uint4*>(xs + xoff(lp, 2 * lq + 1)) = x1;
        __syncthreads();

        // [W_a; W_ga; W_b; W_gb](32 channels each) x x (32 pairs), all scaled
        f32x16_t acc[4];
#pragma unroll
        for (int ob = 0; ob < 4; ++ob)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[ob][r] = 0.f;
        const int bp = lane & 31;
#pragma unroll
        for (int kq = 0; kq < 8; ++kq) {
            const f16x8_t xk = *reinterpret_cast<const f16x8_t*>(xs + xoff(bp, 2 * kq + (lane >> 5)));
#pragma unroll
            for (int ob = 0; ob < 4; ++ob)
                acc[ob] = __builtin_amdgcn_mfma_f32_32x32x16_f16(w[ob][kq], xk, acc[ob], 0, 0, 0);
        }

        // Gate and stage as [c][p] fp32.  Lane holds pair (lane & 31); in
        // register r, channel 32 g + 8 (r / 4) + 4 (lane / 32) + r % 4.
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int c = g * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
            const float ga = __builtin_amdgcn_rcpf(ks.kv_a + __builtin_amdgcn_exp2f(fmaf(acc[1][r], ks.cg_a, ks.sv_a)));
            const float gb2 = __builtin_amdgcn_rcpf(ks.kv_b + __builtin_amdgcn_exp2f(fmaf(acc[3][r], ks.cg_b, ks.sv_b)));
            os[0][c][bp] = ga * acc[0][r];
            os[1][c][bp] = gb2 * acc[2][r];
        }
        __syncthreads();

        // Channel-major stores: 4 lanes write the 32 pairs (64 bytes) of one
        // panel row, one k-step of the blocked layout.  A ragged line's tail
        // writes zeros into the k padding of its step, so every wave issues
        // exactly 4 stores per line.
        const int64_t line_off = panel_off(pg, 0, r0, k0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int ab = i >> 1, c = (t >> 2) + 64 * (i & 1);
            const float4 f0 = *reinterpret_cast<const float4*>(&os[ab][c][8 * (t & 3)]);
            const float4 f1 = *reinterpret_cast<const float4*>(&os[ab][c][8 * (t & 3) + 4]);
            bf16_t* dst = (ab ? B : A) + (line_off + st_lane + 64 * (i & 1) * ch_stride);
            *reinterpret_cast<uint4*>(dst) = make_uint4(pack_bf16x2(f0.x, f0.y), pack_bf16x2(f0.z, f0.w),
                                                        pack_bf16x2(f1.x, f1.y), pack_bf16x2(f1.z, f1.w));
        }
    }
    wait_vmcnt_pinned<0>();   // the ring loads past the last line land before the work-group ends
}

}  // namespace

hipError_t launch_project_mfma(const DeviceWeights& w, const void* z, int64_t ldz, const uint8_t* tmask, int64_t rmoff,
                               int64_t M, int64_t K, int incoming, void* A, void* B, hipStream_t s) {
    const int nch = (int)((K + kP1 - 1) / kP1);
    const int nlines = (int)(M * nch);
    const unsigned g = (unsigned)(nlines < 2 * w.cus ? nlines : 2 * w.cus);
    const int mrange = (int)std::max((K + 31) / 32 * 32, rmoff + (M + 3) / 4 * 4);
    if (incoming)
        hipLaunchKernelGGL((k1_project_mfma<true>), dim3(g), dim3(256), 0, s, (const bf16_t*)z, (int)ldz, tmask,
                           (int)rmoff, mrange, (int)M, (int)K, nlines, w.proj_h, w.ln_in_w_h, w.ln_in_b_h, w.eps,
                           w.k1s, (bf16_t*)A, (bf16_t*)B);
    else
        hipLaunchKernelGGL((k1_project_mfma<false>), dim3(g), dim3(256), 0, s, (const bf16_t*)z, (int)ldz, tmask,
                           (int)rmoff, mrange, (int)M, (int)K, nlines, w.proj_h, w.ln_in_w_h, w.ln_in_b_h, w.eps,
                           w.k1s, (bf16_t*)A, (bf16_t*)B);
    return hipGetLastError();
}

hipError_t launch_project(int dtype, const DeviceWeights& w, const void* z, const uint8_t* mask,
                          int64_t N, int incoming, void* A, void* B, hipStream_t s) {
    const int64_t nchunk = (N + kLine - 1) / kLine;
    const dim3 grid((unsigned)(N * nchunk)), block(256);
    const float4* p4 = reinterpret_cast<const float4*>(w.proj4);
    if (dtype == 0) {
        if (incoming)
            hipLaunchKernelGGL((k1_project_valu<float, true>), grid, block, 0, s, (const float*)z, mask, N,
                               nchunk, p4, w.ln_in_w, w.ln_in_b, w.eps, (float*)A, (float*)B);
        else
            hipLaunchKernelGGL((k1_project_valu<float, false>), grid, block, 0, s, (const float*)z, mask, N,
                               nchunk, p4, w.ln_in_w, w.ln_in_b, w.eps, (float*)A, (float*)B);
    } else {
        hipError_t e = launch_stage_kmask(mask, N, w.kmask_pad, s);
        if (e != hipSuccess) return e;
        return launch_project_mfma(w, z, N, w.kmask_pad, 0, N, N, incoming, A, B, s);
    }
    return hipGetLastError();
}

}  // namespace trimul
