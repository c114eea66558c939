// C ABI of the triangle-multiplication library: argument validation, the
// handle with its repacked weights, and the sequencing of the three kernels
// K1 (projection), K2 (contraction), K3 (epilogue) on the caller's stream.
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <cmath>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "tri_mul.h"
#include "opm.h"
#include "triattn.h"
#include "tri_mul_check.h"
#include "common.h"
#include "kernels.h"

using trimul::DeviceWeights;

struct tri_mul_handle_s {
    int c_z = 0, c = 0, dtype = 0, out_dtype = 0;
    int device = 0;
    DeviceWeights w;
    std::vector<void*> allocations;
};

struct opm_handle_s {
    int d = 0, c_z = 0, out_dtype = 0;
    int device = 0, cus = 256;
    uint16_t* wo = nullptr;   // [c_z][d * d] bf16
    float* bo = nullptr;      // [c_z] fp32
    std::vector<void*> allocations;
};

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

int ok() {
    g_last_error.clear();
    return TRI_MUL_OK;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(TRI_MUL_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t esize(int dtype) { return dtype == TRI_MUL_BF16 ? 2 : 4; }

size_t round256(size_t x) { return (x + 255) & ~size_t(255); }

constexpr int64_t kMaxN = 65536;

// Bytes of the fp32 contraction result in the pair-blocked layout.
size_t result_bytes(int64_t N, int c) { return (size_t)N * (size_t)((N + 31) / 32 * 32) * (size_t)c * 4; }

// Bytes of one blocked operand (all hidden channels) for N tokens.
size_t panel_bytes(int64_t N, int c, int dtype) {
    return (size_t)c * (size_t)trimul::panel_elems(trimul::panel_geom(N, N)) * esize(dtype);
}

// Host conversion of one stored value to double (exact).
double to_double(const unsigned char* p, int dtype) {
    if (dtype == TRI_MUL_F32) {
        float f;
        memcpy(&f, p, 4);
        return f;
    }
    uint16_t h;
    memcpy(&h, p, 2);
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

// Round to the nearest fp16 value, ties to even (subnormals included;
// magnitudes beyond the largest finite value become infinity).
uint16_t to_f16(double v) {
    const uint16_t sign = std::signbit(v) ? 0x8000u : 0u;
    double a = std::fabs(v);
    if (std::isnan(v)) return 0x7e00u;
    if (a >= 65520.0) return sign | 0x7c00u;
    int e;
    std::frexp(a, &e);                      // a = f * 2^e, f in [0.5, 1)
    const int q = std::max(e - 11, -24);    // spacing of fp16 values near a: 2^q
    const double m = std::nearbyint(std::ldexp(a, -q));   // round-half-even (default mode)
    const double r = std::ldexp(m, q);
    if (r == 0) return sign;
    int er;
    std::frexp(r, &er);
    if (er <= -14) return sign | (uint16_t)std::ldexp(r, 24);            // subnormal: r / 2^-24
    const int mant = (int)std::ldexp(r, 11 - er) - 1024;                 // 10 stored bits
    return sign | (uint16_t)(((er - 1 + 15) << 10) | mant);
}

uint16_t to_bf16_exact(double v) {   // v is already a bf16 value
    float f = (float)v;
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

int check_n(int64_t N) {
    if (N < 1 || N > kMaxN) return fail(TRI_MUL_EINVAL, "N = %lld outside [1, %lld]", (long long)N, (long long)kMaxN);
    return TRI_MUL_OK;
}

int check_handle(tri_mul_handle_t h) {
    if (!h) return fail(TRI_MUL_EINVAL, "null handle");
    return TRI_MUL_OK;
}

template <typename T>
int upload(tri_mul_handle_t h, T** dst, const std::vector<T>& src, hipStream_t s) {
    void* p = nullptr;
    hipError_t e = hipMalloc(&p, src.size() * sizeof(T));
    if (e != hipSuccess) return fail(TRI_MUL_ENOMEM, "hipMalloc of %zu bytes: %s", src.size() * sizeof(T), hipGetErrorString(e));
    h->allocations.push_back(p);
    e = hipMemcpyAsync(p, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return hip_fail(e, "weight upload");
    *dst = static_cast<T*>(p);
    return TRI_MUL_OK;
}

void free_all(tri_mul_handle_t h) {
    for (void* p : h->allocations) (void)hipFree(p);
    h->allocations.clear();
}

// K1 and K2 of the full update.  bf16 storage: the projection runs with the
// opposite direction's pair indexing, which writes the direction's operands
// transposed (X_c = A_c^T, the panels tri_mul_project writes for the other
// direction), and the contraction reads both of them transposed -- the same
// sums in the same order, so C is bitwise the one of the plain order, and
// about 4% faster on gfx950 (its LDS stages are unswizzled 2 KB pieces read
// with ds_read_b64_tr_b16).  fp32 storage keeps the plain order (its
// contraction has no transposed reads).  A and B then hold what the layer
// backward's saved form takes.
hipError_t forward_operands_and_contraction(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N,
                                            int incoming, void* A, void* B, float* C, hipStream_t s) {
    if (h->dtype != TRI_MUL_BF16) {
        hipError_t e = trimul::launch_project(h->dtype, h->w, z, mask, N, incoming, A, B, s);
        if (e != hipSuccess) return e;
        return trimul::launch_contract(h->dtype, 1, A, B, C, N, N, N, 0, 0, N, 0, 0, N * N, h->c, 0, nullptr,
                                       h->w.cus, s);
    }
    hipError_t e = trimul::launch_project(h->dtype, h->w, z, mask, N, !incoming, A, B, s);
    if (e != hipSuccess) return e;
    return trimul::launch_contract_transposed(1, 1, A, B, C, N, N, N, h->c, h->w.cus, s);
}

int run_full(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N, void* out, void* ws,
             size_t ws_bytes, void* stream, int incoming) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_n(N)) return rc;
    if (!z || !out || !ws) return fail(TRI_MUL_EINVAL, "null z, out or workspace pointer");
    if (!aligned16(z) || !aligned16(out)) return fail(TRI_MUL_EINVAL, "z and out must be 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(ws) & 255u) return fail(TRI_MUL_EINVAL, "workspace must be 256-byte aligned");
    size_t need = 0;
    if (int rc = tri_mul_workspace_size(h, N, &need)) return rc;
    if (ws_bytes < need) return fail(TRI_MUL_ENOMEM, "workspace of %zu bytes < %zu needed for N = %lld", ws_bytes, need, (long long)N);
    const size_t panel = panel_bytes(N, h->c, h->dtype);
    char* base = static_cast<char*>(ws);
    void* A = base;
    void* B = base + round256(panel);
    float* C = reinterpret_cast<float*>(base + 2 * round256(panel));
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = forward_operands_and_contraction(h, z, mask, N, incoming, A, B, C, s);
    if (e != hipSuccess) return hip_fail(e, "projection or contraction kernel launch");
    trimul::EpilogueArgs ea{C, 1, 0, 0, z, mask, 0, 0, N, N, out};
    e = trimul::launch_epilogue(h->dtype, h->out_dtype, h->w, ea, s);
    if (e != hipSuccess) return hip_fail(e, "epilogue kernel launch");
    return ok();
}

// ------------------------------------------------ no-allocation entry point
//
// Device scratch of tri_mul_update_noalloc: the workspace of the full update
// (A and B panels, fp32 result), kScratchBytes per GPU, held from the
// library's load until the process ends.  Host code never uses the array's
// name as an address: each device's copy is reached through the pointer
// hipGetSymbolAddress returned with that device current (g_scratch).
constexpr size_t kScratchBytes = size_t(256) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// The current device's scratch address, resolved once per device.
int scratch_for(int device, void** ptr) {
    if (device < 0 || device >= kMaxDevices) return fail(TRI_MUL_EUNSUPPORTED, "device %d outside [0, %d)", device, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[device]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "scratch symbol address");
        if (!p) return fail(TRI_MUL_EHIP, "scratch symbol address is null");
        g_scratch[device] = p;
    }
    *ptr = g_scratch[device];
    return TRI_MUL_OK;
}

// Workspace of the layer backward (bf16 path), in this order: A, B and the
// four operands of the contraction backward (panels), C, dA, dB (result
// layout), dx_g [N*N][c_z] fp32, nine unit-block tensors, and the partial
// sums of the weight-gradient reductions.
struct BwdLayout {
    size_t panel, result, dxg, block, part_eb, part_pb, part_w, part_w4, total;
    int grid_pair;   // per-pair stages: one 512-thread work-group per compute unit
    int grid_w;      // weight-gradient sums: two 256-thread work-groups per compute unit
    int grid_w4;     // the four sums over the x blocks: one 512-thread work-group per compute unit
};
BwdLayout bwd_layout(tri_mul_handle_t h, int64_t N) {
    BwdLayout L;
    const int64_t units = N * ((N + 31) / 32);
    L.grid_pair = trimul::backward_grid(units, h->w.cus, 1);
    L.grid_w = trimul::backward_grid(units, h->w.cus, 2);
    L.panel = round256(panel_bytes(N, h->c, h->dtype));
    L.result = round256(result_bytes(N, h->c));
    L.dxg = round256((size_t)N * (size_t)N * (size_t)h->c_z * 4);
    L.block = round256((size_t)units * 128 * 32 * 2);
    L.part_eb = round256((size_t)L.grid_pair * 2 * 128 * 4);
    L.part_pb = round256((size_t)L.grid_pair * 2 * 128 * 4);
    L.part_w = round256((size_t)L.grid_w * 128 * 128 * 4);
    L.grid_w4 = trimul::backward_grid(units, h->w.cus, 1);
    L.part_w4 = round256((size_t)4 * L.grid_w4 * 128 * 128 * 4);
    L.total = 3 * L.panel + 3 * L.result + L.dxg + 9 * L.block + L.part_eb + L.part_pb + L.part_w + L.part_w4;
    return L;
}

int run_backward(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N, const void* dout, void* dz,
                 const tri_mul_grads_t* g, void* ws, size_t ws_bytes, void* stream, int incoming,
                 const void* sA = nullptr, const void* sB = nullptr, const float* sC = nullptr) {
    if (int rc = check_handle(h)) return rc;
    const bool saved = sA || sB || sC;
    if (saved && (!sA || !sB || !sC)) return fail(TRI_MUL_EINVAL, "null saved forward tensor");
    if (saved && (!aligned16(sA) || !aligned16(sB) || !aligned16(sC)))
        return fail(TRI_MUL_EINVAL, "saved forward tensors must be 16-byte aligned");
    if (int rc = check_n(N)) return rc;
    if (h->dtype != TRI_MUL_BF16) return fail(TRI_MUL_EUNSUPPORTED, "the layer backward supports the bf16 storage path only");
    if (!z || !dout || !dz || !g || !ws) return fail(TRI_MUL_EINVAL, "null pointer argument");
    const float* gp[] = {g->ln_in_w, g->ln_in_b, g->w_a, g->w_ga, g->w_b, g->w_gb, g->w_g, g->ln_out_w, g->ln_out_b, g->w_o};
    for (const float* q : gp)
        if (!q) return fail(TRI_MUL_EINVAL, "null gradient pointer");
    if (!aligned16(z) || !aligned16(dout) || !aligned16(dz)) return fail(TRI_MUL_EINVAL, "z, dout and dz must be 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(ws) & 255u) return fail(TRI_MUL_EINVAL, "workspace must be 256-byte aligned");
    const BwdLayout L = bwd_layout(h, N);
    if (ws_bytes < L.total) return fail(TRI_MUL_ENOMEM, "workspace of %zu bytes < %zu needed for N = %lld", ws_bytes, L.total, (long long)N);
    char* p = static_cast<char*>(ws);
    auto take = [&](size_t n) { char* q = p; p += n; return q; };
    const void *A = take(L.panel), *B = take(L.panel);
    void* dCp = take(L.panel);
    const float* C = reinterpret_cast<float*>(take(L.result));
    if (saved) {   // the forward's own A, B, C (their workspace regions go unused)
        A = sA;
        B = sB;
        C = sC;
    }
    float* dA = reinterpret_cast<float*>(take(L.result));
    float* dB = reinterpret_cast<float*>(take(L.result));
    float* dxg = reinterpret_cast<float*>(take(L.dxg));
    trimul::BackwardBlocks bb;
    using trimul::bf16_t;
    bf16_t** blk[] = {&bb.du, &bb.y, &bb.dgg, &bb.xe, &bb.dpa, &bb.dga, &bb.dpb, &bb.dgb, &bb.xp};
    for (bf16_t** q : blk) *q = reinterpret_cast<bf16_t*>(take(L.block));
    float* peb = reinterpret_cast<float*>(take(L.part_eb));
    float* ppb = reinterpret_cast<float*>(take(L.part_pb));
    float* pw = reinterpret_cast<float*>(take(L.part_w));
    float* pw4 = reinterpret_cast<float*>(take(L.part_w4));
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int cus = h->w.cus, G = L.grid_pair, GW = L.grid_w, GW4 = L.grid_w4;

    hipError_t e = hipSuccess;
    if (!saved)   // recompute the forward's operands (stored transposed) and contraction
        e = forward_operands_and_contraction(h, z, mask, N, incoming, const_cast<void*>(A), const_cast<void*>(B),
                                             const_cast<float*>(C), s);
    if (e == hipSuccess) e = trimul::launch_epilogue_backward(h->out_dtype, h->w, C, z, mask, dout, N, dCp, dxg, bb, peb, G, s);
    // A and B hold A^T and B^T: dA = dC B is the plain product of the dC panel
    // with the B^T panel, dB = dC^T A reads dC transposed and A^T as it is
    if (e == hipSuccess)
        e = trimul::launch_contract(h->dtype, 1, dCp, B, dA, N, N, N, 0, 0, N, 0, 0, N * N, h->c, 0, nullptr, cus, s);
    if (e == hipSuccess) e = trimul::launch_contract_transposed(1, 0, dCp, A, dB, N, N, N, h->c, cus, s);
    if (e == hipSuccess) e = trimul::launch_projection_backward(h->w, z, mask, N, incoming, dA, dB, dxg, dz, bb, ppb, G, s);
    const struct { const bf16_t* u; const bf16_t* v; float* out; } wg[] = {{bb.du, bb.y, g->w_o}, {bb.dgg, bb.xe, g->w_g}};
    for (const auto& q : wg) {
        if (e == hipSuccess) e = trimul::launch_wgrad(q.u, q.v, N, pw, GW, s);
        if (e == hipSuccess) e = trimul::launch_sum_parts(pw, GW, 128 * 128, 128 * 128, q.out, s);
    }
    // the four projection weights share the x blocks: one pass over them
    const bf16_t* const u4[4] = {bb.dpa, bb.dga, bb.dpb, bb.dgb};
    float* const out4[4] = {g->w_a, g->w_ga, g->w_b, g->w_gb};
    if (e == hipSuccess) e = trimul::launch_wgrad4(u4, bb.xp, N, pw4, GW4, s);
    for (int o = 0; o < 4; ++o)
        if (e == hipSuccess)
            e = trimul::launch_sum_parts(pw4 + (size_t)o * GW4 * 128 * 128, GW4, 128 * 128, 128 * 128, out4[o], s);
    if (e == hipSuccess) e = trimul::launch_sum_parts(peb, G, 256, 128, g->ln_out_w, s);
    if (e == hipSuccess) e = trimul::launch_sum_parts(peb + 128, G, 256, 128, g->ln_out_b, s);
    if (e == hipSuccess) e = trimul::launch_sum_parts(ppb, G, 256, 128, g->ln_in_w, s);
    if (e == hipSuccess) e = trimul::launch_sum_parts(ppb + 128, G, 256, 128, g->ln_in_b, s);
    if (e != hipSuccess) return hip_fail(e, "backward kernel launch");
    return ok();
}

}  // namespace

extern "C" {

const char* tri_mul_last_error(void) { return g_last_error.c_str(); }

int tri_mul_init(tri_mul_handle_t* out, const tri_mul_params_t* p, void* stream) {
    if (!out || !p) return fail(TRI_MUL_EINVAL, "null handle or params pointer");
    *out = nullptr;
    if (p->dtype != TRI_MUL_F32 && p->dtype != TRI_MUL_BF16) return fail(TRI_MUL_EINVAL, "bad dtype %d", p->dtype);
    if (p->out_dtype != TRI_MUL_F32 && p->out_dtype != TRI_MUL_BF16) return fail(TRI_MUL_EINVAL, "bad out_dtype %d", p->out_dtype);
    if (p->c_z <= 0 || p->c <= 0) return fail(TRI_MUL_EINVAL, "c_z = %d, c = %d must be positive", p->c_z, p->c);
    if (p->c_z != 128 || p->c != 128) return fail(TRI_MUL_EUNSUPPORTED, "only c_z = c = 128 is supported (got %d, %d)", p->c_z, p->c);
    if (!(p->ln_eps > 0.f)) return fail(TRI_MUL_EINVAL, "ln_eps must be positive");
    const void* ptrs[] = {p->ln_in_w, p->ln_in_b, p->w_a, p->w_ga, p->w_b, p->w_gb, p->w_g, p->ln_out_w, p->ln_out_b, p->w_o};
    for (const void* q : ptrs)
        if (!q) return fail(TRI_MUL_EINVAL, "null weight pointer");

    tri_mul_handle_t h = new (std::nothrow) tri_mul_handle_s;
    if (!h) return fail(TRI_MUL_ENOMEM, "host allocation failed");
    h->c_z = p->c_z;
    h->c = p->c;
    h->dtype = p->dtype;
    h->out_dtype = p->out_dtype;
    h->w.eps = p->ln_eps;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipGetDevice(&h->device);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&h->w.cus, hipDeviceAttributeMultiprocessorCount, h->device);
    if (e != hipSuccess) {
        delete h;
        return hip_fail(e, "device query");
    }
    void* scr = nullptr;   // the no-allocation entry point's scratch on this device
    if (int rc = scratch_for(h->device, &scr)) {
        delete h;
        return rc;
    }

    const int cz = p->c_z, c = p->c;
    const size_t es = esize(p->dtype);
    auto fetch = [&](const void* src, size_t n, std::vector<double>& dst) -> int {
        std::vector<unsigned char> raw(n * es);
        hipError_t err = hipMemcpyAsync(raw.data(), src, n * es, hipMemcpyDeviceToHost, s);
        if (err == hipSuccess) err = hipStreamSynchronize(s);
        if (err != hipSuccess) return hip_fail(err, "weight download");
        dst.resize(n);
        for (size_t i = 0; i < n; ++i) dst[i] = to_double(raw.data() + i * es, p->dtype);
        return TRI_MUL_OK;
    };
    std::vector<double> lnw, lnb, wa, wga, wb, wgb, wg, low, lob, wo;
    int rc = TRI_MUL_OK;
    if (!rc) rc = fetch(p->ln_in_w, cz, lnw);
    if (!rc) rc = fetch(p->ln_in_b, cz, lnb);
    if (!rc) rc = fetch(p->w_a, (size_t)c * cz, wa);
    if (!rc) rc = fetch(p->w_ga, (size_t)c * cz, wga);
    if (!rc) rc = fetch(p->w_b, (size_t)c * cz, wb);
    if (!rc) rc = fetch(p->w_gb, (size_t)c * cz, wgb);
    if (!rc) rc = fetch(p->w_g, (size_t)cz * cz, wg);
    if (!rc) rc = fetch(p->ln_out_w, c, low);
    if (!rc) rc = fetch(p->ln_out_b, c, lob);
    if (!rc) rc = fetch(p->w_o, (size_t)cz * c, wo);
    if (rc) {
        delete h;
        return rc;
    }

    // fp32 copies for the VALU kernels.
    std::vector<float> f_lnw(lnw.begin(), lnw.end()), f_lnb(lnb.begin(), lnb.end());
    std::vector<float> f_low(low.begin(), low.end()), f_lob(lob.begin(), lob.end());
    std::vector<float> proj4((size_t)cz * c * 4), wo_t((size_t)c * cz), wg_t((size_t)cz * cz);
    for (int d = 0; d < cz; ++d)
        for (int ch = 0; ch < c; ++ch) {
            float* q = &proj4[((size_t)d * c + ch) * 4];
            q[0] = (float)wa[(size_t)ch * cz + d];
            q[1] = (float)wga[(size_t)ch * cz + d];
            q[2] = (float)wb[(size_t)ch * cz + d];
            q[3] = (float)wgb[(size_t)ch * cz + d];
        }
    for (int d = 0; d < cz; ++d)
        for (int ch = 0; ch < c; ++ch) wo_t[(size_t)ch * cz + d] = (float)wo[(size_t)d * c + ch];
    for (int d = 0; d < cz; ++d)
        for (int e2 = 0; e2 < cz; ++e2) wg_t[(size_t)e2 * cz + d] = (float)wg[(size_t)d * cz + e2];

    if (!rc) rc = upload(h, &h->w.ln_in_w, f_lnw, s);
    if (!rc) rc = upload(h, &h->w.ln_in_b, f_lnb, s);
    if (!rc) rc = upload(h, &h->w.ln_out_w, f_low, s);
    if (!rc) rc = upload(h, &h->w.ln_out_b, f_lob, s);
    if (!rc) rc = upload(h, &h->w.proj4, proj4, s);
    if (!rc) rc = upload(h, &h->w.wo_t, wo_t, s);
    if (!rc) rc = upload(h, &h->w.wg_t, wg_t, s);
    if (!rc) {
        std::vector<uint8_t> zeros((size_t)trimul::kMaskStageBytes, 0);
        rc = upload(h, &h->w.kmask_pad, zeros, s);
    }
    if (!rc && p->dtype == TRI_MUL_BF16) {
        // MFMA operand copies: projection rows grouped per 32 hidden channels
        // (W_a, W_ga, W_b, W_gb blocks), then W_o and W_g rows.
        std::vector<uint16_t> pb((size_t)4 * c * cz), eb((size_t)2 * cz * 128);
        for (int g = 0; g < c / 32; ++g)
            for (int m = 0; m < 4; ++m)
                for (int r = 0; r < 32; ++r) {
                    const std::vector<double>& src = m == 0 ? wa : m == 1 ? wga : m == 2 ? wb : wgb;
                    const size_t row = (size_t)g * 128 + m * 32 + r;
                    for (int d = 0; d < cz; ++d) pb[row * cz + d] = to_bf16_exact(src[(size_t)(g * 32 + r) * cz + d]);
                }
        for (int d = 0; d < cz; ++d)
            for (int k = 0; k < 128; ++k) {
                eb[(size_t)d * 128 + k] = to_bf16_exact(wo[(size_t)d * c + k]);
                eb[(size_t)(cz + d) * 128 + k] = to_bf16_exact(wg[(size_t)d * cz + k]);
            }
        // backward: W_o^T and W_g^T rows; row d of [W_a^T | W_ga^T | W_b^T | W_gb^T]
        std::vector<uint16_t> ebt((size_t)256 * cz), pbt((size_t)cz * 4 * c);
        for (int k = 0; k < 128; ++k)
            for (int d = 0; d < cz; ++d) {
                ebt[(size_t)k * cz + d] = to_bf16_exact(wo[(size_t)d * c + k]);
                ebt[(size_t)(128 + k) * cz + d] = to_bf16_exact(wg[(size_t)d * cz + k]);
            }
        for (int d = 0; d < cz; ++d)
            for (int m = 0; m < 4; ++m) {
                const std::vector<double>& src = m == 0 ? wa : m == 1 ? wga : m == 2 ? wb : wgb;
                for (int ch = 0; ch < c; ++ch) pbt[((size_t)d * 4 + m) * c + ch] = to_bf16_exact(src[(size_t)ch * cz + d]);
            }
        // fp16 projection operands with power-of-two scales: |x| <= sqrt(c_z - 1)
        // max|gamma| + max|beta| after LayerNorm, and each weight matrix's
        // largest entry, both brought into [2^14, 2^15] (scales clamped to
        // 2^-40 .. 2^40; operands that would still exceed the fp16 range
        // are refused).
        auto pow2_scale = [](double bound) -> int {
            if (!(bound > 0)) return 0;
            int s2 = (int)std::floor(std::log2(32768.0 / bound));
            return std::max(-40, std::min(40, s2));
        };
        double gmax = 0, bmax = 0;
        for (int d = 0; d < cz; ++d) gmax = std::max(gmax, std::fabs(lnw[d])), bmax = std::max(bmax, std::fabs(lnb[d]));
        const double xbound = std::sqrt((double)cz - 1.0) * gmax + bmax;
        const int sx = pow2_scale(xbound);
        int sw[4];
        for (int m = 0; m < 4; ++m) {
            const std::vector<double>& src = m == 0 ? wa : m == 1 ? wga : m == 2 ? wb : wgb;
            double mx = 0;
            for (double v2 : src) mx = std::max(mx, std::fabs(v2));
            sw[m] = pow2_scale(mx);
            if (mx * std::ldexp(1.0, sw[m]) > 65504.0) rc = fail(TRI_MUL_EUNSUPPORTED, "projection weights beyond the supported range");
        }
        if (xbound * std::ldexp(1.0, sx) > 65504.0) rc = fail(TRI_MUL_EUNSUPPORTED, "input LayerNorm parameters beyond the supported range");
        std::vector<uint16_t> ph((size_t)4 * c * cz);
        for (int g = 0; g < c / 32; ++g)
            for (int m = 0; m < 4; ++m)
                for (int r = 0; r < 32; ++r) {
                    const std::vector<double>& src = m == 0 ? wa : m == 1 ? wga : m == 2 ? wb : wgb;
                    const size_t row = (size_t)g * 128 + m * 32 + r;
                    for (int d = 0; d < cz; ++d) ph[row * cz + d] = to_f16(std::ldexp(src[(size_t)(g * 32 + r) * cz + d], sw[m]));
                }
        std::vector<float> lnw_h(cz), lnb_h(cz);
        for (int d = 0; d < cz; ++d) lnw_h[d] = (float)std::ldexp(lnw[d], sx), lnb_h[d] = (float)std::ldexp(lnb[d], sx);
        const double log2e = 1.4426950408889634;
        auto& k = h->w.k1s;
        k.kv_a = (float)std::ldexp(1.0, sx + sw[0]);
        k.cg_a = (float)(-log2e * std::ldexp(1.0, -(sx + sw[1])));
        k.sv_a = (float)(sx + sw[0]);
        k.kv_b = (float)std::ldexp(1.0, sx + sw[2]);
        k.cg_b = (float)(-log2e * std::ldexp(1.0, -(sx + sw[3])));
        k.sv_b = (float)(sx + sw[2]);
        if (!rc) rc = upload(h, &h->w.proj_h, ph, s);
        if (!rc) rc = upload(h, &h->w.ln_in_w_h, lnw_h, s);
        if (!rc) rc = upload(h, &h->w.ln_in_b_h, lnb_h, s);
        if (!rc) rc = upload(h, &h->w.proj_bf, pb, s);
        if (!rc) rc = upload(h, &h->w.epi_bf, eb, s);
        if (!rc) rc = upload(h, &h->w.epit_bf, ebt, s);
        if (!rc) rc = upload(h, &h->w.projt_bf, pbt, s);
    }
    if (!rc) {
        e = hipStreamSynchronize(s);
        if (e != hipSuccess) rc = hip_fail(e, "init synchronisation");
    }
    if (rc) {
        free_all(h);
        delete h;
        return rc;
    }
    *out = h;
    return ok();
}

int tri_mul_destroy(tri_mul_handle_t h) {
    if (!h) return ok();
    hipError_t e = hipDeviceSynchronize();
    free_all(h);
    delete h;
    if (e != hipSuccess) return hip_fail(e, "destroy synchronisation");
    return ok();
}

int tri_mul_workspace_size(tri_mul_handle_t h, int64_t N, size_t* bytes) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_n(N)) return rc;
    if (!bytes) return fail(TRI_MUL_EINVAL, "null bytes pointer");
    *bytes = 2 * round256(panel_bytes(N, h->c, h->dtype)) + round256(result_bytes(N, h->c));
    return ok();
}

int tri_mul_panel_size(tri_mul_handle_t h, int64_t N, size_t* bytes) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_n(N)) return rc;
    if (!bytes) return fail(TRI_MUL_EINVAL, "null bytes pointer");
    *bytes = panel_bytes(N, h->c, h->dtype);
    return ok();
}

int tri_mul_outgoing(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N, void* out, void* ws,
                     size_t ws_bytes, void* stream) {
    return run_full(h, z, mask, N, out, ws, ws_bytes, stream, 0);
}

int tri_mul_incoming(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N, void* out, void* ws,
                     size_t ws_bytes, void* stream) {
    return run_full(h, z, mask, N, out, ws, ws_bytes, stream, 1);
}

int tri_mul_update_noalloc(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N, int32_t direction,
                           void* out, void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (direction != TRI_MUL_OUTGOING && direction != TRI_MUL_INCOMING) return fail(TRI_MUL_EINVAL, "bad direction %d", direction);
    if (int rc = check_n(N)) return rc;
    size_t need = 0;
    if (int rc = tri_mul_workspace_size(h, N, &need)) return rc;
    if (need > kScratchBytes)
        return fail(TRI_MUL_EUNSUPPORTED, "N = %lld needs %zu bytes of workspace; the no-allocation scratch holds %zu",
                    (long long)N, need, kScratchBytes);
    int device = 0;
    const hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_fail(e, "device query");
    void* ws = nullptr;
    if (int rc = scratch_for(device, &ws)) return rc;
    return run_full(h, z, mask, N, out, ws, kScratchBytes, stream, direction);
}

int tri_mul_project(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N, int32_t direction,
                    void* a_panels, void* b_panels, void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_n(N)) return rc;
    if (direction != TRI_MUL_OUTGOING && direction != TRI_MUL_INCOMING) return fail(TRI_MUL_EINVAL, "bad direction %d", direction);
    if (!z || !a_panels || !b_panels) return fail(TRI_MUL_EINVAL, "null z or panel pointer");
    if (!aligned16(z) || !aligned16(a_panels) || !aligned16(b_panels)) return fail(TRI_MUL_EINVAL, "z and panels must be 16-byte aligned");
    hipError_t e = trimul::launch_project(h->dtype, h->w, z, mask, N, direction, a_panels, b_panels, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "projection kernel launch");
    return ok();
}

int tri_mul_contract(tri_mul_handle_t h, const void* a_panels, const void* b_panels, int64_t N, float* c_out,
                     void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_n(N)) return rc;
    if (!a_panels || !b_panels || !c_out) return fail(TRI_MUL_EINVAL, "null panel or output pointer");
    if (!aligned16(a_panels) || !aligned16(b_panels) || !aligned16(c_out)) return fail(TRI_MUL_EINVAL, "panels and output must be 16-byte aligned");
    hipError_t e = trimul::launch_contract(h->dtype, 1, a_panels, b_panels, c_out, N, N, N, 0, 0, N, 0, 0, N * N, h->c,
                                           0, nullptr, h->w.cus, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "contraction kernel launch");
    return ok();
}

int tri_mul_contract_transposed(tri_mul_handle_t h, const void* at_panels, const void* bt_panels, int64_t N,
                                float* c_out, void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_n(N)) return rc;
    if (h->dtype != TRI_MUL_BF16) return fail(TRI_MUL_EUNSUPPORTED, "transposed operands exist for the bf16 storage path only");
    if (!at_panels || !bt_panels || !c_out) return fail(TRI_MUL_EINVAL, "null panel or output pointer");
    if (!aligned16(at_panels) || !aligned16(bt_panels) || !aligned16(c_out))
        return fail(TRI_MUL_EINVAL, "panels and output must be 16-byte aligned");
    hipError_t e = trimul::launch_contract_transposed(1, 1, at_panels, bt_panels, c_out, N, N, N, h->c, h->w.cus,
                                                      static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "contraction kernel launch");
    return ok();
}

int tri_mul_epilogue(tri_mul_handle_t h, const float* c_in, const void* z, const uint8_t* mask, int64_t N, void* out,
                     void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_n(N)) return rc;
    if (!c_in || !z || !out) return fail(TRI_MUL_EINVAL, "null C, z or out pointer");
    if (!aligned16(c_in) || !aligned16(z) || !aligned16(out)) return fail(TRI_MUL_EINVAL, "C, z and out must be 16-byte aligned");
    trimul::EpilogueArgs ea{c_in, 1, 0, 0, z, mask, 0, 0, N, N, out};
    hipError_t e = trimul::launch_epilogue(h->dtype, h->out_dtype, h->w, ea, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "epilogue kernel launch");
    return ok();
}

int tri_mul_contract_backward_workspace_size(tri_mul_handle_t h, int64_t N, size_t* bytes) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_n(N)) return rc;
    if (!bytes) return fail(TRI_MUL_EINVAL, "null bytes pointer");
    // bf16: dC as a panel; fp32 also the transposes of dC, A and B
    *bytes = (h->dtype == TRI_MUL_BF16 ? 1 : 4) * round256(panel_bytes(N, h->c, h->dtype));
    return ok();
}

int tri_mul_contract_backward(tri_mul_handle_t h, const float* dC, const void* a_panels, const void* b_panels,
                              int64_t N, float* dA, float* dB, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_n(N)) return rc;
    if (!dC || !a_panels || !b_panels || !dA || !dB || !ws) return fail(TRI_MUL_EINVAL, "null pointer argument");
    if (!aligned16(dC) || !aligned16(a_panels) || !aligned16(b_panels) || !aligned16(dA) || !aligned16(dB))
        return fail(TRI_MUL_EINVAL, "tensors must be 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(ws) & 255u) return fail(TRI_MUL_EINVAL, "workspace must be 256-byte aligned");
    size_t need = 0;
    if (int rc = tri_mul_contract_backward_workspace_size(h, N, &need)) return rc;
    if (ws_bytes < need) return fail(TRI_MUL_ENOMEM, "workspace of %zu bytes < %zu needed for N = %lld", ws_bytes, need, (long long)N);
    const size_t panel = round256(panel_bytes(N, h->c, h->dtype));
    char* base = static_cast<char*>(ws);
    void* dCp = base;               // dC as operand rows i, k = j
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int cus = h->w.cus;
    hipError_t e = trimul::launch_result_to_panel(h->dtype, dC, dCp, N, cus, s);
    if (h->dtype == TRI_MUL_BF16) {
        // dA[i][k] = sum_j dC[i][j] B[j][k];  dB[j][k] = sum_i dC[i][j] A[i][k]: the matrix
        // cores read B, dC and A transposed from their panels
        if (e == hipSuccess) e = trimul::launch_contract_transposed(0, 1, dCp, b_panels, dA, N, N, N, h->c, cus, s);
        if (e == hipSuccess) e = trimul::launch_contract_transposed(1, 1, dCp, a_panels, dB, N, N, N, h->c, cus, s);
        if (e != hipSuccess) return hip_fail(e, "backward contraction kernel launch");
        return ok();
    }
    void* dCt = base + panel;       // dC^T: rows j, k = i
    void* At = base + 2 * panel;    // A^T
    void* Bt = base + 3 * panel;    // B^T
    if (e == hipSuccess) e = trimul::launch_panel_transpose(h->dtype, dCp, dCt, N, cus, s);
    if (e == hipSuccess) e = trimul::launch_panel_transpose(h->dtype, a_panels, At, N, cus, s);
    if (e == hipSuccess) e = trimul::launch_panel_transpose(h->dtype, b_panels, Bt, N, cus, s);
    if (e != hipSuccess) return hip_fail(e, "backward layout kernel launch");
    // dA[i][k] = sum_j dC[i][j] B^T[k][j];  dB[j][k] = sum_i dC^T[j][i] A^T[k][i]
    e = trimul::launch_contract(h->dtype, 1, dCp, Bt, dA, N, N, N, 0, 0, N, 0, 0, N * N, h->c, 0, nullptr, cus, s);
    if (e == hipSuccess)
        e = trimul::launch_contract(h->dtype, 1, dCt, At, dB, N, N, N, 0, 0, N, 0, 0, N * N, h->c, 0, nullptr, cus, s);
    if (e != hipSuccess) return hip_fail(e, "backward contraction kernel launch");
    return ok();
}

}  // extern "C"

namespace {

// Checks of a block view's sizes, ranges and panel strides, shared by the
// block entry points.
int check_view(const tri_mul_block_view_t* v) {
    if (!v) return fail(TRI_MUL_EINVAL, "null view");
    if (v->n_total < 1 || v->rows < 1 || v->cols < 1 || v->klen < 1) return fail(TRI_MUL_EINVAL, "empty or negative view sizes");
    if (v->row0 < 0 || v->col0 < 0 || v->k0 < 0 || v->row0 + v->rows > v->n_total || v->col0 + v->cols > v->n_total ||
        v->k0 + v->klen > v->n_total)
        return fail(TRI_MUL_EINVAL, "view ranges exceed n_total = %lld", (long long)v->n_total);
    if (v->rows > kMaxN || v->cols > kMaxN || v->klen > trimul::kMaxKPanel)
        return fail(TRI_MUL_EUNSUPPORTED, "tile sides and k-panel length are limited to %lld", (long long)kMaxN);
    if (v->ld_a < v->klen || v->ld_b < v->klen || (v->ld_a % 8) || (v->ld_b % 8))
        return fail(TRI_MUL_EINVAL, "ld_a / ld_b must be >= klen and multiples of 8");
    // the kernels address a 256-row panel tile with 32-bit byte offsets
    if (v->ld_a > kMaxN || v->ld_b > kMaxN)
        return fail(TRI_MUL_EUNSUPPORTED, "ld_a / ld_b are limited to %lld elements", (long long)kMaxN);
    if (v->k_count < 1 || v->k_index < 0 || v->k_index >= v->k_count) return fail(TRI_MUL_EINVAL, "bad k_index %d / k_count %d", v->k_index, v->k_count);
    return TRI_MUL_OK;
}

// Pointer checks of a ring step: panels (or the workspace holding them
// repacked), accumulator, and on the last k-panel the tile's z and output.
int check_block(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* a_panel, const void* b_panel,
                const float* acc, const void* z_tile, const void* out_tile) {
    (void)h;
    if (int rc = check_view(v)) return rc;
    if (!a_panel || !b_panel || !acc) return fail(TRI_MUL_EINVAL, "null panel or accumulator pointer");
    if (!aligned16(a_panel) || !aligned16(b_panel) || !aligned16(acc)) return fail(TRI_MUL_EINVAL, "panels and accumulator must be 16-byte aligned");
    const bool last = v->k_index == v->k_count - 1;
    if (last) {
        if (!z_tile || !out_tile) return fail(TRI_MUL_EINVAL, "the last k-panel needs z_tile and out_tile");
        if (!aligned16(z_tile) || !aligned16(out_tile)) return fail(TRI_MUL_EINVAL, "z_tile and out_tile must be 16-byte aligned");
    }
    return TRI_MUL_OK;
}

// Bytes of the two repacked panels (blocked layout), each 256-byte aligned.
size_t block_ws_a(const tri_mul_block_view_t* v) {
    const size_t nk = (size_t)((v->klen + 31) / 32);
    return round256((size_t)128 * (size_t)((v->rows + 255) / 256) * nk * 256 * 32 * 2);
}
size_t block_ws_b(const tri_mul_block_view_t* v) {
    const size_t nk = (size_t)((v->klen + 31) / 32);
    return round256((size_t)128 * (size_t)((v->cols + 255) / 256) * nk * 256 * 32 * 2);
}
// Bytes of the staged k-mask kept at the end of the workspace (0/1 per k,
// zero-padded to a multiple of 32), so that a repack on one stream never
// shares staging with an epilogue on another.
size_t block_ws_m(const tri_mul_block_view_t* v) { return round256((size_t)((v->klen + 31) / 32 * 32)); }
size_t block_ws_total(const tri_mul_block_view_t* v) { return block_ws_a(v) + block_ws_b(v) + block_ws_m(v); }

// Validation shared by the repacking entry points: the view's sizes, and a
// workspace of block_ws_total bytes, 256-byte aligned.
int check_block_ws(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* ws, size_t ws_bytes) {
    if (h->dtype != TRI_MUL_BF16) return fail(TRI_MUL_EUNSUPPORTED, "repacked panels exist for the bf16 storage path only");
    if (!ws) return fail(TRI_MUL_EINVAL, "null workspace");
    if (reinterpret_cast<uintptr_t>(ws) & 255u) return fail(TRI_MUL_EINVAL, "workspace must be 256-byte aligned");
    const size_t need = block_ws_total(v);
    if (ws_bytes < need) return fail(TRI_MUL_ENOMEM, "workspace of %zu bytes, %zu needed", ws_bytes, need);
    return TRI_MUL_OK;
}

// Stage the view's k-mask into the workspace and repack both panels.
hipError_t block_repack(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* a_panel, const void* b_panel,
                        const uint8_t* mask, void* ws, hipStream_t s) {
    char* wa = static_cast<char*>(ws);
    char* wb = wa + block_ws_a(v);
    uint8_t* km = reinterpret_cast<uint8_t*>(wb + block_ws_b(v));
    hipError_t e = trimul::launch_stage_kmask(mask ? mask + v->k0 : nullptr, v->klen, km, s);
    if (e == hipSuccess) e = trimul::launch_panel_block(a_panel, v->rows, v->ld_a, v->klen, h->c, km, wa, s);
    if (e == hipSuccess) e = trimul::launch_panel_block(b_panel, v->cols, v->ld_b, v->klen, h->c, km, wb, s);
    return e;
}

}  // namespace

extern "C" {

int tri_mul_block_accumulate(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* a_panel,
                             const void* b_panel, float* acc, const uint8_t* mask, const void* z_tile,
                             void* out_tile, void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_block(h, v, a_panel, b_panel, acc, z_tile, out_tile)) return rc;
    const bool last = v->k_index == v->k_count - 1;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t sA = v->rows * v->ld_a, sB = v->cols * v->ld_b, sC = v->rows * v->cols;
    hipError_t e = hipSuccess;
    const uint8_t* kmask = nullptr;
    if (mask) {   // the kernels read the k-range of the mask as a zero-padded 0/1 copy
        e = trimul::launch_stage_kmask(mask + v->k0, v->klen, h->w.kmask_pad, s);
        if (e != hipSuccess) return hip_fail(e, "mask staging kernel launch");
        kmask = h->w.kmask_pad;
    }
    e = trimul::launch_contract(h->dtype, 0, a_panel, b_panel, acc, v->rows, v->cols, v->klen, v->ld_a, v->ld_b,
                                v->cols, sA, sB, sC, h->c, v->k_index > 0, kmask, h->w.cus, s);
    if (e != hipSuccess) return hip_fail(e, "contraction kernel launch");
    if (last) {
        trimul::EpilogueArgs ea{acc, 0, v->cols, sC, z_tile, mask, v->row0, v->col0, v->rows, v->cols, out_tile};
        e = trimul::launch_epilogue(h->dtype, h->out_dtype, h->w, ea, s);
        if (e != hipSuccess) return hip_fail(e, "epilogue kernel launch");
    }
    return ok();
}


int tri_mul_block_workspace_size(tri_mul_handle_t h, const tri_mul_block_view_t* v, size_t* bytes) {
    if (int rc = check_handle(h)) return rc;
    if (!v || !bytes) return fail(TRI_MUL_EINVAL, "null view or bytes pointer");
    if (v->rows < 1 || v->cols < 1 || v->klen < 1 || v->rows > kMaxN || v->cols > kMaxN ||
        v->klen > trimul::kMaxKPanel)
        return fail(TRI_MUL_EINVAL, "tile sides and k-panel length must lie in [1, %lld]", (long long)kMaxN);
    *bytes = h->dtype == TRI_MUL_BF16 ? block_ws_total(v) : 0;
    return ok();
}

int tri_mul_block_accumulate_ws(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* a_panel,
                                const void* b_panel, float* acc, const uint8_t* mask, const void* z_tile,
                                void* out_tile, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_block(h, v, a_panel, b_panel, acc, z_tile, out_tile)) return rc;
    if (h->dtype != TRI_MUL_BF16)   // the fp32 path has no blocked form: the plain call is the same op
        return tri_mul_block_accumulate(h, v, a_panel, b_panel, acc, mask, z_tile, out_tile, stream);
    if (int rc = check_block_ws(h, v, ws, ws_bytes)) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* wa = static_cast<char*>(ws);
    char* wb = wa + block_ws_a(v);
    const bool last = v->k_index == v->k_count - 1;
    hipError_t e = block_repack(h, v, a_panel, b_panel, mask, ws, s);
    if (e != hipSuccess) return hip_fail(e, "panel repack kernel launch");
    e = trimul::launch_contract_blocked_rowc(wa, wb, acc, v->rows, v->cols, v->klen, h->c, v->k_index > 0, h->w.cus, s);
    if (e != hipSuccess) return hip_fail(e, "contraction kernel launch");
    if (last) {
        const int64_t sC = v->rows * v->cols;
        trimul::EpilogueArgs ea{acc, 0, v->cols, sC, z_tile, mask, v->row0, v->col0, v->rows, v->cols, out_tile};
        e = trimul::launch_epilogue(h->dtype, h->out_dtype, h->w, ea, s);
        if (e != hipSuccess) return hip_fail(e, "epilogue kernel launch");
    }
    return ok();
}

int tri_mul_block_accumulator_size(tri_mul_handle_t h, const tri_mul_block_view_t* v, size_t* bytes) {
    if (int rc = check_handle(h)) return rc;
    if (!v || !bytes) return fail(TRI_MUL_EINVAL, "null view or bytes pointer");
    if (v->rows < 1 || v->cols < 1 || v->rows > kMaxN || v->cols > kMaxN)
        return fail(TRI_MUL_EINVAL, "tile sides must lie in [1, %lld]", (long long)kMaxN);
    *bytes = (size_t)v->rows * (size_t)((v->cols + 31) / 32 * 32) * (size_t)h->c * 4;
    return ok();
}

int tri_mul_block_repack(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* a_panel,
                         const void* b_panel, const uint8_t* mask, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_view(v)) return rc;
    if (!a_panel || !b_panel) return fail(TRI_MUL_EINVAL, "null panel pointer");
    if (!aligned16(a_panel) || !aligned16(b_panel)) return fail(TRI_MUL_EINVAL, "panels must be 16-byte aligned");
    if (int rc = check_block_ws(h, v, ws, ws_bytes)) return rc;
    hipError_t e = block_repack(h, v, a_panel, b_panel, mask, ws, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "panel repack kernel launch");
    return ok();
}

int tri_mul_block_accumulate_packed(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* ws,
                                    size_t ws_bytes, float* acc, const uint8_t* mask, const void* z_tile,
                                    void* out_tile, int32_t reserve_cus, void* stream) {
    if (int rc = check_handle(h)) return rc;
    // the panels live in ws: pass ws in their place for the shared checks
    if (int rc = check_block(h, v, ws, ws, acc, z_tile, out_tile)) return rc;
    if (int rc = check_block_ws(h, v, ws, ws_bytes)) return rc;
    if (reserve_cus < 0 || reserve_cus > h->w.cus - 8)
        return fail(TRI_MUL_EINVAL, "reserve_cus = %d outside [0, %d]", reserve_cus, h->w.cus - 8);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const char* wa = static_cast<const char*>(ws);
    const char* wb = wa + block_ws_a(v);
    const int cus = (h->w.cus - reserve_cus) & ~7;   // whole XCD groups
    hipError_t e = trimul::launch_contract_blocked_packed(wa, wb, acc, v->rows, v->cols, v->klen, h->c,
                                                          v->k_index > 0, cus, s);
    if (e != hipSuccess) return hip_fail(e, "contraction kernel launch");
    if (v->k_index == v->k_count - 1) {
        trimul::EpilogueArgs ea{acc, 1, 0, 0, z_tile, mask, v->row0, v->col0, v->rows, v->cols, out_tile};
        e = trimul::launch_epilogue(h->dtype, h->out_dtype, h->w, ea, s);
        if (e != hipSuccess) return hip_fail(e, "epilogue kernel launch");
    }
    return ok();
}

int tri_mul_block_panel_size(tri_mul_handle_t h, int64_t rows, int64_t klen, size_t* bytes) {
    if (int rc = check_handle(h)) return rc;
    if (!bytes) return fail(TRI_MUL_EINVAL, "null bytes pointer");
    if (h->dtype != TRI_MUL_BF16) return fail(TRI_MUL_EUNSUPPORTED, "blocked panels exist for the bf16 storage path only");
    if (rows < 1 || klen < 1) return fail(TRI_MUL_EINVAL, "empty or negative panel sizes");
    if (rows > kMaxN || klen > trimul::kMaxKPanel)
        return fail(TRI_MUL_EUNSUPPORTED, "panel sides are limited to %lld", (long long)kMaxN);
    *bytes = (size_t)h->c * (size_t)((rows + 255) / 256) * (size_t)((klen + 31) / 32) * 256 * 32 * 2;
    return ok();
}

int tri_mul_block_project(tri_mul_handle_t h, const void* z_tile, int64_t ld_z, const uint8_t* mask, int64_t n_total,
                          int64_t row0, int64_t col0, int64_t rows, int64_t cols, int32_t direction, void* a_panel,
                          void* b_panel, void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (h->dtype != TRI_MUL_BF16) return fail(TRI_MUL_EUNSUPPORTED, "blocked panels exist for the bf16 storage path only");
    if (direction != TRI_MUL_OUTGOING && direction != TRI_MUL_INCOMING) return fail(TRI_MUL_EINVAL, "bad direction %d", direction);
    if (!z_tile || !a_panel || !b_panel) return fail(TRI_MUL_EINVAL, "null z_tile or panel pointer");
    if (!aligned16(z_tile) || !aligned16(a_panel) || !aligned16(b_panel))
        return fail(TRI_MUL_EINVAL, "z_tile and the panels must be 16-byte aligned");
    if (n_total < 1 || rows < 1 || cols < 1) return fail(TRI_MUL_EINVAL, "empty or negative tile sizes");
    if (row0 < 0 || col0 < 0 || row0 + rows > n_total || col0 + cols > n_total)
        return fail(TRI_MUL_EINVAL, "tile ranges exceed n_total = %lld", (long long)n_total);
    if (rows > trimul::kMaxKPanel || cols > trimul::kMaxKPanel)
        return fail(TRI_MUL_EUNSUPPORTED, "tile sides are limited to %lld", (long long)trimul::kMaxKPanel);
    if (ld_z < cols) return fail(TRI_MUL_EINVAL, "ld_z = %lld < cols = %lld", (long long)ld_z, (long long)cols);
    // the projection addresses 32 pairs of a tile column with 32-bit byte offsets
    if (ld_z > kMaxN) return fail(TRI_MUL_EUNSUPPORTED, "ld_z is limited to %lld pairs", (long long)kMaxN);
    hipStream_t s = static_cast<hipStream_t>(stream);
    // operand rows i and contraction index k: the tile's rows and columns
    // (outgoing) or its columns and rows (incoming)
    const bool in = direction == TRI_MUL_INCOMING;
    const int64_t m0 = in ? col0 : row0, M = in ? cols : rows, k0 = in ? row0 : col0, K = in ? rows : cols;
    hipError_t e = trimul::launch_stage_tile_mask(mask, m0, M, k0, K, h->w.kmask_pad, s);
    if (e == hipSuccess)
        e = trimul::launch_project_mfma(h->w, z_tile, ld_z, h->w.kmask_pad, (K + 31) / 32 * 32, M, K, in ? 1 : 0,
                                        a_panel, b_panel, s);
    if (e != hipSuccess) return hip_fail(e, "projection kernel launch");
    return ok();
}

int tri_mul_block_accumulate_blocked(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* a_panel,
                                     const void* b_panel, float* acc, const uint8_t* mask, const void* z_tile,
                                     void* out_tile, int32_t reserve_cus, void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (h->dtype != TRI_MUL_BF16) return fail(TRI_MUL_EUNSUPPORTED, "blocked panels exist for the bf16 storage path only");
    if (!v) return fail(TRI_MUL_EINVAL, "null view");
    tri_mul_block_view_t w = *v;   // the strides of row-major panels do not apply
    w.ld_a = w.ld_b = (v->klen + 7) / 8 * 8;
    if (int rc = check_block(h, &w, a_panel, b_panel, acc, z_tile, out_tile)) return rc;
    if (reserve_cus < 0 || reserve_cus > h->w.cus - 8)
        return fail(TRI_MUL_EINVAL, "reserve_cus = %d outside [0, %d]", reserve_cus, h->w.cus - 8);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int cus = (h->w.cus - reserve_cus) & ~7;   // whole XCD groups
    hipError_t e = trimul::launch_contract_blocked_packed(a_panel, b_panel, acc, v->rows, v->cols, v->klen, h->c,
                                                          v->k_index > 0, cus, s);
    if (e != hipSuccess) return hip_fail(e, "contraction kernel launch");
    if (v->k_index == v->k_count - 1) {
        trimul::EpilogueArgs ea{acc, 1, 0, 0, z_tile, mask, v->row0, v->col0, v->rows, v->cols, out_tile};
        e = trimul::launch_epilogue(h->dtype, h->out_dtype, h->w, ea, s);
        if (e != hipSuccess) return hip_fail(e, "epilogue kernel launch");
    }
    return ok();
}

int tri_mul_block_accumulate_transposed(tri_mul_handle_t h, const tri_mul_block_view_t* v, const void* at_panel,
                                        const void* bt_panel, float* acc, const uint8_t* mask, const void* z_tile,
                                        void* out_tile, int32_t reserve_cus, void* stream) {
    if (int rc = check_handle(h)) return rc;
    if (h->dtype != TRI_MUL_BF16) return fail(TRI_MUL_EUNSUPPORTED, "blocked panels exist for the bf16 storage path only");
    if (!v) return fail(TRI_MUL_EINVAL, "null view");
    tri_mul_block_view_t w = *v;   // the strides of row-major panels do not apply
    w.ld_a = w.ld_b = (v->klen + 7) / 8 * 8;
    if (int rc = check_block(h, &w, at_panel, bt_panel, acc, z_tile, out_tile)) return rc;
    if (reserve_cus < 0 || reserve_cus > h->w.cus - 8)
        return fail(TRI_MUL_EINVAL, "reserve_cus = %d outside [0, %d]", reserve_cus, h->w.cus - 8);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int cus = (h->w.cus - reserve_cus) & ~7;   // whole XCD groups
    hipError_t e = trimul::launch_contract_transposed(1, 1, at_panel, bt_panel, acc, v->rows, v->cols, v->klen, h->c,
                                                      cus, s, v->k_index > 0);
    if (e != hipSuccess) return hip_fail(e, "contraction kernel launch");
    if (v->k_index == v->k_count - 1) {
        trimul::EpilogueArgs ea{acc, 1, 0, 0, z_tile, mask, v->row0, v->col0, v->rows, v->cols, out_tile};
        e = trimul::launch_epilogue(h->dtype, h->out_dtype, h->w, ea, s);
        if (e != hipSuccess) return hip_fail(e, "epilogue kernel launch");
    }
    return ok();
}

int tri_mul_backward_workspace_size(tri_mul_handle_t h, int64_t N, size_t* bytes) {
    if (int rc = check_handle(h)) return rc;
    if (int rc = check_n(N)) return rc;
    if (!bytes) return fail(TRI_MUL_EINVAL, "null bytes pointer");
    *bytes = bwd_layout(h, N).total;
    return ok();
}

int tri_mul_outgoing_backward(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N, const void* dout,
                              void* dz, const tri_mul_grads_t* grads, void* ws, size_t ws_bytes, void* stream) {
    return run_backward(h, z, mask, N, dout, dz, grads, ws, ws_bytes, stream, 0);
}

int tri_mul_incoming_backward(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N, const void* dout,
                              void* dz, const tri_mul_grads_t* grads, void* ws, size_t ws_bytes, void* stream) {
    return run_backward(h, z, mask, N, dout, dz, grads, ws, ws_bytes, stream, 1);
}

int tri_mul_outgoing_backward_saved(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N,
                                    const void* a_panels, const void* b_panels, const float* c_result,
                                    const void* dout, void* dz, const tri_mul_grads_t* grads, void* ws,
                                    size_t ws_bytes, void* stream) {
    if (!a_panels || !b_panels || !c_result) return fail(TRI_MUL_EINVAL, "null saved forward tensor");
    return run_backward(h, z, mask, N, dout, dz, grads, ws, ws_bytes, stream, 0, a_panels, b_panels, c_result);
}

int tri_mul_incoming_backward_saved(tri_mul_handle_t h, const void* z, const uint8_t* mask, int64_t N,
                                    const void* a_panels, const void* b_panels, const float* c_result,
                                    const void* dout, void* dz, const tri_mul_grads_t* grads, void* ws,
                                    size_t ws_bytes, void* stream) {
    if (!a_panels || !b_panels || !c_result) return fail(TRI_MUL_EINVAL, "null saved forward tensor");
    return run_backward(h, z, mask, N, dout, dz, grads, ws, ws_bytes, stream, 1, a_panels, b_panels, c_result);
}

}  // extern "C"

// ---------------------------------------------------------------- outer product mean

namespace {

constexpr int64_t kOpmMaxTile = 2048;    // tokens per tile side: rows * d <= 65536 contraction rows
constexpr int64_t kOpmMaxSeq = 65536;    // sequences per step

size_t opm_panel_bytes(int64_t rows, int64_t K) {
    return round256((size_t)trimul::panel_elems(trimul::panel_geom(rows, K)) * 2);
}
size_t opm_sum_bytes(int64_t rows, int64_t cols) { return round256((size_t)rows * 32 * (size_t)cols * 32 * 4); }
size_t opm_cnt_bytes(int64_t rows, int64_t cols) { return round256((size_t)rows * (size_t)((cols + 31) / 32 * 32) * 4); }

int opm_check(opm_handle_t h) { return h ? TRI_MUL_OK : fail(TRI_MUL_EINVAL, "null handle"); }

}  // namespace

extern "C" {

int opm_init(opm_handle_t* out, const opm_params_t* p, void* stream) {
    if (!out || !p) return fail(TRI_MUL_EINVAL, "null handle or params pointer");
    *out = nullptr;
    if (p->out_dtype != TRI_MUL_F32 && p->out_dtype != TRI_MUL_BF16) return fail(TRI_MUL_EINVAL, "bad out_dtype %d", p->out_dtype);
    if (p->d <= 0 || p->c_z <= 0) return fail(TRI_MUL_EINVAL, "d = %d, c_z = %d must be positive", p->d, p->c_z);
    if (p->d != 32 || p->c_z != 128) return fail(TRI_MUL_EUNSUPPORTED, "only d = 32, c_z = 128 is supported (got %d, %d)", p->d, p->c_z);
    if (!p->w_o) return fail(TRI_MUL_EINVAL, "null w_o");
    opm_handle_t h = new (std::nothrow) opm_handle_s;
    if (!h) return fail(TRI_MUL_ENOMEM, "host allocation failed");
    h->d = p->d;
    h->c_z = p->c_z;
    h->out_dtype = p->out_dtype;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipGetDevice(&h->device);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&h->cus, hipDeviceAttributeMultiprocessorCount, h->device);
    const size_t nw = (size_t)h->c_z * h->d * h->d;
    std::vector<uint16_t> bias_raw(h->c_z, 0);
    if (e == hipSuccess && p->b_o) e = hipMemcpyAsync(bias_raw.data(), p->b_o, h->c_z * 2, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    int rc = e == hipSuccess ? TRI_MUL_OK : hip_fail(e, "opm init");
    std::vector<float> bias(h->c_z);
    for (int i = 0; i < h->c_z; ++i) bias[i] = (float)to_double(reinterpret_cast<unsigned char*>(&bias_raw[i]), TRI_MUL_BF16);
    void* pw = nullptr;
    if (!rc) {
        e = hipMalloc(&pw, nw * 2);
        if (e != hipSuccess) rc = fail(TRI_MUL_ENOMEM, "hipMalloc of %zu bytes: %s", nw * 2, hipGetErrorString(e));
        else h->allocations.push_back(pw);
    }
    if (!rc) {
        e = hipMemcpyAsync(pw, p->w_o, nw * 2, hipMemcpyDeviceToDevice, s);
        if (e != hipSuccess) rc = hip_fail(e, "w_o copy");
        h->wo = static_cast<uint16_t*>(pw);
    }
    void* pb = nullptr;
    if (!rc) {
        e = hipMalloc(&pb, h->c_z * 4);
        if (e != hipSuccess) rc = fail(TRI_MUL_ENOMEM, "hipMalloc of %d bytes: %s", h->c_z * 4, hipGetErrorString(e));
        else h->allocations.push_back(pb);
    }
    if (!rc) {
        e = hipMemcpyAsync(pb, bias.data(), h->c_z * 4, hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) rc = hip_fail(e, "b_o upload");
        h->bo = static_cast<float*>(pb);
    }
    if (rc) {
        for (void* q : h->allocations) (void)hipFree(q);
        delete h;
        return rc;
    }
    *out = h;
    return ok();
}

int opm_destroy(opm_handle_t h) {
    if (!h) return ok();
    hipError_t e = hipDeviceSynchronize();
    for (void* q : h->allocations) (void)hipFree(q);
    delete h;
    if (e != hipSuccess) return hip_fail(e, "destroy synchronisation");
    return ok();
}

int opm_accumulator_size(opm_handle_t h, int64_t rows, int64_t cols, size_t* bytes) {
    if (int rc = opm_check(h)) return rc;
    if (!bytes) return fail(TRI_MUL_EINVAL, "null bytes pointer");
    if (rows < 1 || cols < 1 || rows > kOpmMaxTile || cols > kOpmMaxTile)
        return fail(TRI_MUL_EINVAL, "tile %lld x %lld outside [1, %lld]^2", (long long)rows, (long long)cols, (long long)kOpmMaxTile);
    *bytes = opm_sum_bytes(rows, cols) + opm_cnt_bytes(rows, cols);
    return ok();
}

int opm_workspace_size(opm_handle_t h, int64_t rows, int64_t cols, int64_t slen, size_t* bytes) {
    if (int rc = opm_check(h)) return rc;
    if (!bytes) return fail(TRI_MUL_EINVAL, "null bytes pointer");
    if (rows < 1 || cols < 1 || rows > kOpmMaxTile || cols > kOpmMaxTile)
        return fail(TRI_MUL_EINVAL, "tile %lld x %lld outside [1, %lld]^2", (long long)rows, (long long)cols, (long long)kOpmMaxTile);
    if (slen < 1 || slen > kOpmMaxSeq) return fail(TRI_MUL_EINVAL, "slen = %lld outside [1, %lld]", (long long)slen, (long long)kOpmMaxSeq);
    // the sums' operands transposed (slen rows, tokens * 32 columns), the counts' plain
    *bytes = opm_panel_bytes(slen, rows * 32) + opm_panel_bytes(slen, cols * 32) + opm_panel_bytes(rows, slen) +
             opm_panel_bytes(cols, slen);
    return ok();
}

int opm_block_accumulate(opm_handle_t h, const opm_block_view_t* v, const void* a, const void* b,
                         const uint8_t* mask, float* acc, void* out_tile, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = opm_check(h)) return rc;
    if (!v) return fail(TRI_MUL_EINVAL, "null view");
    if (!a || !b || !acc || !ws) return fail(TRI_MUL_EINVAL, "null a, b, accumulator or workspace pointer");
    if (v->n_total < 1 || v->s_total < 1 || v->rows < 1 || v->cols < 1 || v->slen < 1 || v->row0 < 0 || v->col0 < 0 ||
        v->s0 < 0 || v->row0 + v->rows > v->n_total || v->col0 + v->cols > v->n_total || v->s0 + v->slen > v->s_total)
        return fail(TRI_MUL_EINVAL, "view outside the %lld tokens x %lld sequences", (long long)v->n_total, (long long)v->s_total);
    if (v->k_count < 1 || v->k_index < 0 || v->k_index >= v->k_count)
        return fail(TRI_MUL_EINVAL, "bad k_index %d / k_count %d", v->k_index, v->k_count);
    size_t need = 0;
    if (int rc = opm_workspace_size(h, v->rows, v->cols, v->slen, &need)) return rc;
    if (ws_bytes < need) return fail(TRI_MUL_ENOMEM, "workspace of %zu bytes < %zu needed", ws_bytes, need);
    if (!aligned16(a) || !aligned16(b) || !aligned16(acc)) return fail(TRI_MUL_EINVAL, "a, b and the accumulator must be 16-byte aligned");
    if (reinterpret_cast<uintptr_t>(ws) & 255u) return fail(TRI_MUL_EINVAL, "workspace must be 256-byte aligned");
    const bool last = v->k_index == v->k_count - 1;
    if (last && (!out_tile || !aligned16(out_tile))) return fail(TRI_MUL_EINVAL, "the last step needs a 16-byte aligned out_tile");
    char* p = static_cast<char*>(ws);
    void* PA = p;
    p += opm_panel_bytes(v->slen, v->rows * 32);
    void* PB = p;
    p += opm_panel_bytes(v->slen, v->cols * 32);
    void* MA = p;
    p += opm_panel_bytes(v->rows, v->slen);
    void* MB = p;
    float* sums = acc;
    float* cnt = reinterpret_cast<float*>(reinterpret_cast<char*>(acc) + opm_sum_bytes(v->rows, v->cols));
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = trimul::launch_opm_pack(a, mask, v->n_total, v->row0, v->rows, v->s0, v->slen, PA, MA, s);
    if (e == hipSuccess) e = trimul::launch_opm_pack(b, mask, v->n_total, v->col0, v->cols, v->s0, v->slen, PB, MB, s);
    if (e != hipSuccess) return hip_fail(e, "pack kernel launch");
    const int accumulate = v->k_index > 0;
    e = trimul::launch_contract_transposed(1, 1, PA, PB, sums, v->rows * 32, v->cols * 32, v->slen, 1, h->cus, s,
                                           accumulate);
    if (e == hipSuccess)
        e = trimul::launch_contract(TRI_MUL_BF16, 1, MA, MB, cnt, v->rows, v->cols, v->slen, 0, 0, 0, 0, 0, 0, 1,
                                    accumulate, nullptr, h->cus, s);
    if (e != hipSuccess) return hip_fail(e, "contraction kernel launch");
    if (last) {
        e = trimul::launch_opm_epilogue(h->out_dtype == TRI_MUL_BF16, sums, cnt, v->rows, v->cols, h->wo, h->bo,
                                        out_tile, h->cus, s);
        if (e != hipSuccess) return hip_fail(e, "epilogue kernel launch");
    }
    return ok();
}

int opm_forward_workspace_size(opm_handle_t h, int64_t S, int64_t N, size_t* bytes) {
    if (int rc = opm_check(h)) return rc;
    if (!bytes) return fail(TRI_MUL_EINVAL, "null bytes pointer");
    size_t accb = 0, wsb = 0;
    if (int rc = opm_accumulator_size(h, N, N, &accb)) return rc;
    if (int rc = opm_workspace_size(h, N, N, S, &wsb)) return rc;
    *bytes = accb + wsb;
    return ok();
}

int opm_forward(opm_handle_t h, const void* a, const void* b, const uint8_t* mask, int64_t S, int64_t N,
                void* out, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = opm_check(h)) return rc;
    if (!ws) return fail(TRI_MUL_EINVAL, "null workspace pointer");
    size_t need = 0, accb = 0;
    if (int rc = opm_forward_workspace_size(h, S, N, &need)) return rc;
    if (ws_bytes < need) return fail(TRI_MUL_ENOMEM, "workspace of %zu bytes < %zu needed", ws_bytes, need);
    if (int rc = opm_accumulator_size(h, N, N, &accb)) return rc;
    const opm_block_view_t v{N, S, 0, N, 0, N, 0, S, 0, 1};
    return opm_block_accumulate(h, &v, a, b, mask, static_cast<float*>(ws), out, static_cast<char*>(ws) + accb,
                                ws_bytes - accb, stream);
}

}  // extern "C"

// ---------------------------------------------------------------- triangle attention core

namespace {

constexpr int64_t kTaMaxN = 16384;

int ta_check(const tri_attn_view_t* v) {
    if (!v) return fail(TRI_MUL_EINVAL, "null view");
    if (v->rows < 1 || v->n < 1 || v->n > kTaMaxN) return fail(TRI_MUL_EINVAL, "rows = %lld, n = %lld outside [1, inf) x [1, %lld]", (long long)v->rows, (long long)v->n, (long long)kTaMaxN);
    if (v->heads < 1 || v->heads > 16) return fail(TRI_MUL_EINVAL, "heads = %d outside [1, 16]", v->heads);
    if (v->rows * (int64_t)v->heads * ((v->n + 127) / 128) > (int64_t)INT32_MAX) return fail(TRI_MUL_EUNSUPPORTED, "too many rows");
    if (v->out_dtype != TRI_MUL_F32 && v->out_dtype != TRI_MUL_BF16) return fail(TRI_MUL_EINVAL, "bad out_dtype %d", v->out_dtype);
    if (v->ld_bias < v->n || (v->ld_bias % 8)) return fail(TRI_MUL_EINVAL, "ld_bias = %lld must be >= n and a multiple of 8", (long long)v->ld_bias);
    if (v->k0 < 0 || v->klen < 1 || v->k0 + v->klen > v->n || (v->k0 % 8)) return fail(TRI_MUL_EINVAL, "key range [%lld, +%lld) must lie in [0, n) with k0 %% 8 == 0", (long long)v->k0, (long long)v->klen);
    if (v->k_count < 1 || v->k_index < 0 || v->k_index >= v->k_count) return fail(TRI_MUL_EINVAL, "bad k_index %d / k_count %d", v->k_index, v->k_count);
    if (v->ld_bias > (int64_t)1 << 22) return fail(TRI_MUL_EUNSUPPORTED, "ld_bias = %lld above 2^22", (long long)v->ld_bias);
    return TRI_MUL_OK;
}

size_t ta_sum_elems(const tri_attn_view_t* v) { return (size_t)v->rows * v->n * v->heads * 32; }
size_t ta_ml_elems(const tri_attn_view_t* v) { return (size_t)v->rows * v->heads * v->n; }

}  // namespace

extern "C" {

int tri_attn_state_size(const tri_attn_view_t* v, size_t* bytes) {
    if (int rc = ta_check(v)) return rc;
    if (!bytes) return fail(TRI_MUL_EINVAL, "null bytes pointer");
    *bytes = (ta_sum_elems(v) + 2 * ta_ml_elems(v)) * 4;
    return ok();
}

int tri_attn_chunk(const tri_attn_view_t* v, const void* q, const void* k, const void* vv, const void* bias,
                   const uint8_t* mask, float* state, void* out, void* stream) {
    if (int rc = ta_check(v)) return rc;
    if (!q || !k || !vv || !bias) return fail(TRI_MUL_EINVAL, "null q, k, v or bias pointer");
    const bool last = v->k_index == v->k_count - 1;
    const bool single = v->k_count == 1;
    if (!single && !state) return fail(TRI_MUL_EINVAL, "a chunked attention needs a state");
    if (last && !out) return fail(TRI_MUL_EINVAL, "the last step needs out");
    if (!aligned16(q) || !aligned16(k) || !aligned16(vv) || !aligned16(bias) || (state && !aligned16(state)) ||
        (out && !aligned16(out)))
        return fail(TRI_MUL_EINVAL, "tensors must be 16-byte aligned");
    float* stA = state;
    float* stM = state ? state + ta_sum_elems(v) : nullptr;
    float* stL = state ? stM + ta_ml_elems(v) : nullptr;
    hipError_t e = trimul::launch_triattn(v->out_dtype == TRI_MUL_BF16, q, k, vv, bias, mask, v->rows, v->n,
                                          v->heads, v->ld_bias, v->k0, v->k0 + v->klen, stA, stM, stL,
                                          v->k_index > 0, last, out, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "attention kernel launch");
    return ok();
}

int tri_attn_forward(const void* q, const void* k, const void* v, const void* bias, const uint8_t* mask,
                     int64_t rows, int64_t n, int32_t heads, int64_t ld_bias, int32_t out_dtype, void* out,
                     void* stream) {
    const tri_attn_view_t view{rows, n, heads, out_dtype, ld_bias, 0, n, 0, 1};
    return tri_attn_chunk(&view, q, k, v, bias, mask, nullptr, out, stream);
}

int tri_mul_check_contract_loads(int a_mode, int b_mode, int64_t M, int64_t N, int64_t K, int64_t lda,
                                 int64_t ldb, int64_t a_stride, int64_t b_stride, int batch, uint64_t a_bytes,
                                 uint64_t b_bytes, int grid, int all_channels, tri_mul_load_check_t* out) {
    if (!out) return fail(TRI_MUL_EINVAL, "null out");
    if (M < 1 || N < 1 || K < 1 || batch < 1 || grid < 1 || M > kMaxN || N > kMaxN || K > kMaxN)
        return fail(TRI_MUL_EINVAL, "sizes must lie in [1, %lld]", (long long)kMaxN);
    for (int m : {a_mode, b_mode})
        if (m < TRI_MUL_OPERAND_BLOCKED || m > TRI_MUL_OPERAND_TRANSPOSED) return fail(TRI_MUL_EINVAL, "bad operand mode %d", m);
    if ((a_mode == TRI_MUL_OPERAND_ROW_MAJOR && (lda < K || lda % 8 || lda > kMaxN)) ||
        (b_mode == TRI_MUL_OPERAND_ROW_MAJOR && (ldb < K || ldb % 8 || ldb > kMaxN)))
        return fail(TRI_MUL_EINVAL, "row-major ld must be >= K, <= %lld and a multiple of 8", (long long)kMaxN);
    trimul::K2CheckCounts n;
    trimul::k2_check_loads(a_mode, b_mode, M, N, K, lda, ldb, a_stride, b_stride, batch, a_bytes, b_bytes, grid,
                           all_channels, n);
    *out = tri_mul_load_check_t{n.tiles, n.loads, n.elems, n.bad_tiles, n.bad_desc, n.bad_elem};
    return ok();
}

int tri_mul_check_contract_result(int64_t M, int64_t N, int batch, uint64_t c_bytes, int all_channels,
                                  tri_mul_load_check_t* out) {
    if (!out) return fail(TRI_MUL_EINVAL, "null out");
    if (M < 1 || N < 1 || batch < 1 || M > kMaxN || N > kMaxN)
        return fail(TRI_MUL_EINVAL, "sizes must lie in [1, %lld]", (long long)kMaxN);
    trimul::K2CheckCounts n;
    trimul::k2_check_c(M, N, batch, c_bytes, all_channels, n);
    *out = tri_mul_load_check_t{n.tiles, n.loads, n.elems, n.bad_tiles, n.bad_desc, n.bad_elem};
    return ok();
}

}  // extern "C"
