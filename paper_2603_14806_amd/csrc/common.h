// Device-side helpers shared by the triangle-multiplication kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace trimul {

constexpr int kCz = 128;   // pair channels c_z supported by the kernels
constexpr int kCh = 128;   // hidden channels c supported by the kernels

typedef uint16_t bf16_t;   // raw bfloat16 storage

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(bf16_t v) { return __uint_as_float((uint32_t)v << 16); }

// Round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16_t f2bf(float f) {
    __bf16 b = (__bf16)f;
    return __builtin_bit_cast(bf16_t, b);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats to two round-to-nearest-even bf16 in one dword (lo in bits 0-15);
// one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const f32x2_t f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

// Sum over each aligned group of 8 lanes, returned to all 8 lanes, with DPP
// moves instead of LDS permutes: pairs (xor 1), quads (xor 2), then the two
// quads of the group (lane i meets lane 7 - i).  Every lane of a group adds
// the same operands, so all 8 results are bitwise equal.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float sum_lanes8(float v) {
    v += dpp_mov<0xb1>(v);    // quad_perm [1, 0, 3, 2]
    v += dpp_mov<0x4e>(v);    // quad_perm [2, 3, 0, 1]
    v += dpp_mov<0x141>(v);   // row_half_mirror
    return v;
}
__device__ __forceinline__ float sum_lanes4(float v) {
    v += dpp_mov<0xb1>(v);
    v += dpp_mov<0x4e>(v);
    return v;
}

template <typename T> struct Store;
template <> struct Store<float> {
    static __device__ __forceinline__ float ld(const float* p) { return *p; }
    static __device__ __forceinline__ void st(float* p, float v) { *p = v; }
};
template <> struct Store<bf16_t> {
    static __device__ __forceinline__ float ld(const bf16_t* p) { return bf2f(*p); }
    static __device__ __forceinline__ void st(bf16_t* p, float v) { *p = f2bf(v); }
};

// Blocked layout of the contraction operands ("panels") written by the
// projection and read by the contraction: for hidden channel c, operand row i
// and contraction index k, the element lives at
//     ((c * tiles_r + i / 256) * ksteps + k / 32) * (256 * 32) + (i % 256) * 32 + k % 32
// with tiles_r = ceil(rows / 256) and ksteps = ceil(K / 32), so that one
// 256-row x 32-k step of a contraction tile is one contiguous 16 KB block.
constexpr int kBlkRows = 256, kBlkK = 32;
struct PanelGeom {
    int64_t tiles_r;   // ceil(rows / 256)
    int64_t ksteps;    // ceil(K / 32)
};
__host__ __device__ __forceinline__ PanelGeom panel_geom(int64_t rows, int64_t K) {
    return PanelGeom{(rows + kBlkRows - 1) / kBlkRows, (K + kBlkK - 1) / kBlkK};
}
__host__ __device__ __forceinline__ int64_t panel_elems(const PanelGeom& g) {
    return g.tiles_r * g.ksteps * kBlkRows * kBlkK;   // per channel
}
__host__ __device__ __forceinline__ int64_t panel_off(const PanelGeom& g, int64_t c, int64_t i, int64_t k) {
    return ((c * g.tiles_r + i / kBlkRows) * g.ksteps + k / kBlkK) * (kBlkRows * kBlkK) + (i % kBlkRows) * kBlkK +
           k % kBlkK;
}

// Pair-blocked layout of the fp32 contraction result C written by the
// contraction and read by the epilogue (full update and stage calls): element
// (channel c, row i, column j) of nch channels lives at
//     ((i * ceil(cols / 32) + j / 32) * nch + c) * 32 + j % 32
// so that the 128 channels of 32 consecutive pairs of a row are one
// contiguous 16 KB block.
constexpr int kResJ = 32;
__host__ __device__ __forceinline__ int64_t result_off(int64_t jblocks, int nch, int64_t c, int64_t i, int64_t j) {
    return ((i * jblocks + j / kResJ) * nch + c) * kResJ + j % kResJ;
}

// Logistic function with the hardware exponential and reciprocal (v_exp_f32,
// v_rcp_f32, ~1 ulp each) instead of an IEEE division; exp overflow gives
// rcp(inf) = 0 as the limit requires.
__device__ __forceinline__ float sigmoidf_(float t) { return __builtin_amdgcn_rcpf(1.0f + __expf(-t)); }

// Raw buffer resource over `bytes` bytes starting at p: loads at offsets
// >= bytes return zero (the hardware range check of untyped buffer access).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// ---------------------------------------------------------------- direct-to-LDS

typedef int v4i_t __attribute__((ext_vector_type(4)));

// Raw buffer descriptor (gfx9): base, stride 0, num_records = bytes, 32-bit
// untyped access.  Loads at byte offsets >= bytes return zero.  The
// arguments must be wave-uniform; the words are moved to scalar registers
// explicitly because the inline-assembly loads take the descriptor there.
__device__ __forceinline__ v4i_t buffer_desc(const void* p, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(p);
    v4i_t r;
    r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r.y = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
    r.z = __builtin_amdgcn_readfirstlane((int)bytes);
    r.w = 0x00020000;
    return r;
}

// Direct-to-LDS load: lane i writes `size` bytes at LDS address lds + size * i.
// Issued as inline assembly so that the compiler does not serialise every
// later LDS read behind it; the kernel waits on vmcnt itself.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_load16(v4i_t r, uint32_t voff, uint32_t soff, uint32_t lds) {
    lds = __builtin_amdgcn_readfirstlane(lds);
    soff = __builtin_amdgcn_readfirstlane(soff);
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :: "s"(lds), "v"(voff), "s"(r), "s"(soff) : "memory", "m0");
}
__device__ __forceinline__ void lds_load4(v4i_t r, uint32_t voff, uint32_t soff, uint32_t lds) {
    lds = __builtin_amdgcn_readfirstlane(lds);
    soff = __builtin_amdgcn_readfirstlane(soff);
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, %3 offen lds"
                 :: "s"(lds), "v"(voff), "s"(r), "s"(soff) : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return __builtin_amdgcn_readfirstlane((uint32_t)reinterpret_cast<uintptr_t>(p));
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// The same wait as inline assembly with a memory clobber: the compiler moves
// no load or store across it, so the number of vector-memory instructions
// issued between a load and its wait is the one the source shows.
template <int N>
__device__ __forceinline__ void wait_vmcnt_pinned() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}

}  // namespace trimul
