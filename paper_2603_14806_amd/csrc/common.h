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

__device__ __forceinline__ float sigmoidf_(float t) { return 1.0f / (1.0f + __expf(-t)); }

// Raw buffer resource over `bytes` bytes starting at p: loads at offsets
// >= bytes return zero (the hardware range check of untyped buffer access).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

}  // namespace trimul
