// gfx950 kernels of the sparse INT8 linear layer, and their launchers.
//
// Method (Section "Sparse GEMM operators", Figure 1, Algorithm 1): the stored
// 4x1 weight blocks are broadcast into one operand of an int8 dot-product
// instruction, the input columns named by the weight's mask are picked out of
// the dense input ("re-organised"), products accumulate in int32, and bias and
// the other post-operators are applied once per output before the store.
//
// MI355X mapping:
//  * The weight operand is the A operand of v_smfmac_i32_16x16x128_i8, the
//    4:2-sparse int8 matrix-core instruction: 16 output channels (4
//    block-rows) x one 128-column window, at most 2 stored values per row in
//    every aligned group of 4 columns, each with a 2-bit column index. The
//    packer turns the block mask into these indices, so the matrix core
//    itself selects the input columns the mask names. Groups where a
//    block-row stores 3-4 blocks use a second (slot 1) operand on the window.
//  * A workgroup of WM x WN waves owns TM tokens x NT 16-channel tiles. Per
//    128-column window it copies its TM x 128 input bytes (row-major, 16-byte
//    row pad: the B operand is two conflict-free ds_read_b128 per lane) and
//    its NT weight operands (plus any overflow operands) into LDS with direct
//    global->LDS loads; each wave reads its operands into registers, starts
//    the next window's copies into the other buffer, then issues its matrix
//    instructions, so copies overlap the math.
//  * After the last window the epilogue (dequantise, bias, GELU(erf),
//    requantise) runs on the int32 accumulators in registers; each lane holds
//    the 4 channels of one block-row for one token and stores them together.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <memory>
#include <string>
#include <type_traits>

#include "sl_internal.h"

namespace sl {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int kXs = kWin + 16;        // LDS bytes per staged token row (pad: conflict-free B reads)
constexpr int kXRowPieces = kXs / 16; // 16-byte pieces per staged row, the last one padding
constexpr int kXcds = 8;              // accelerator complex dies, each with its own L2
constexpr size_t kLdsMax = 160 * 1024; // LDS per workgroup on gfx950

#define HIP_TRY(expr)                                                                     \
    do {                                                                                  \
        hipError_t e_ = (expr);                                                           \
        if (e_ != hipSuccess) {                                                           \
            set_error(std::string(#expr) + ": " + hipGetErrorString(e_));                 \
            return SL_ERR_HIP;                                                            \
        }                                                                                 \
    } while (0)

struct LinearArgs {
    const int8_t *x;
    void *y;
    int64_t m;
    int32_t n;
    int32_t k;
    const int8_t *main;
    const int8_t *ovf;
    const uint32_t *ovf_ptr;
    const float *w_scale;
    const float *bias;
    float sx;
    float inv_so;
    int32_t n_tiles;
    int32_t n_win;
    int32_t n_cgroups;  // channel groups of NT tiles
};

// Workgroup shape: WM x WN waves; a wave owns ST 16-token subtiles x CT
// 16-channel tiles; D windows are in flight (D LDS buffers). One window's
// buffer is a flat run of 16-byte pieces: the TM staged token rows (9 pieces
// each, the 9th padding), then NT main operands, then up to NT overflow
// operands (68 pieces each). Each region is padded to a whole number of
// 64-lane copy instructions per wave, so every wave issues the same fixed
// number of copies per window and waits can count them.
template <int ST, int CT, int WM, int WN, int D>
struct Shape {
    static constexpr int NW = WM * WN;
    static constexpr int NTH = 64 * NW;
    static constexpr int TM = 16 * ST * WM;  // tokens per workgroup
    static constexpr int NT = CT * WN;       // channel tiles per workgroup
    static constexpr int CX = (TM * kXRowPieces + NTH - 1) / NTH;  // copies per wave: token rows
    static constexpr int CA = (NT * kOpPieces + NTH - 1) / NTH;    // copies per wave: operands
    static constexpr int XP = CX * NTH;
    static constexpr int AP = CA * NTH;
    static constexpr int COPIES = CX + 2 * CA;  // per wave per window
    static constexpr int BUF = (XP + 2 * AP) * 16;
    static constexpr int LDS = D * BUF;
};

// internal kind: GELU + requantisation evaluated with erf (no usable table)
constexpr int kEpiI8GeluErf = 5;

// The GELU + requantisation step table, passed by value to the kernel of
// SL_EPI_I8_GELU.
struct GeluArg {
    float hinv, off;
    int32_t nc, pad;
    GeluCell cell[kGeluCells];
};

// Workgroups are dispatched round-robin over the XCDs. Renumber them so that
// each XCD runs a contiguous range of work items; adjacent work items share a
// token tile, so that tile's rows are fetched into one L2.
__device__ __forceinline__ int64_t xcd_work_index(int64_t bid, int64_t nwg)
{
    const int64_t q = nwg / kXcds, r = nwg % kXcds;
    const int64_t x = bid % kXcds, j = bid / kXcds;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

// GELU, erf form, in the same fp32 operation order as the definition.
__device__ __forceinline__ float gelu_erf(float y)
{
#pragma clang fp contract(off)
    const float t = y * 0.70710678118654752f;
    const float e = erff(t);
    const float h = 0.5f * y;
    const float one_e = 1.0f + e;
    return h * one_e;
}

__device__ __forceinline__ int32_t requant_i8(float g, float inv_so)
{
#pragma clang fp contract(off)
    const float v = g * inv_so;
    float r = __builtin_rintf(v);
    r = fminf(fmaxf(r, -127.0f), 127.0f);
    return (int32_t)r;
}

template <int KIND>
__device__ __forceinline__ void epilogue_store(const LinearArgs &a, const i32x4 acc, int64_t tok, int32_t ch0,
                                               const float s[4], const float b[4], const GeluCell *tab,
                                               float hinv, float off, float cmax)
{
#pragma clang fp contract(off)
    if (tok >= a.m) return;
    const int64_t off64 = tok * a.n + ch0;
    if constexpr (KIND == SL_EPI_ACC_I32) {
        *reinterpret_cast<i32x4 *>(static_cast<int32_t *>(a.y) + off64) = acc;
    } else if constexpr (KIND == SL_EPI_I8_GELU) {
        uint32_t packed = 0;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float y = (float)acc[r] * s[r];
            y = y + b[r];
            const float c = __builtin_amdgcn_fmed3f(__builtin_fmaf(y, hinv, off), 0.0f, cmax);
            const GeluCell e = tab[(int)c];
            const int q = y >= e.thr ? e.q_hi : e.q_lo;
            packed |= ((uint32_t)q & 0xffu) << (8 * r);
        }
        *reinterpret_cast<uint32_t *>(static_cast<int8_t *>(a.y) + off64) = packed;
    } else {
        float g[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float y = (float)acc[r] * s[r];
            y = y + b[r];
            g[r] = (KIND == SL_EPI_F32_GELU || KIND == kEpiI8GeluErf) ? gelu_erf(y) : y;
        }
        if constexpr (KIND == SL_EPI_F32 || KIND == SL_EPI_F32_GELU) {
            *reinterpret_cast<float4 *>(static_cast<float *>(a.y) + off64) = make_float4(g[0], g[1], g[2], g[3]);
        } else {
            uint32_t packed = 0;
#pragma unroll
            for (int r = 0; r < 4; ++r) packed |= ((uint32_t)requant_i8(g[r], a.inv_so) & 0xffu) << (8 * r);
            *reinterpret_cast<uint32_t *>(static_cast<int8_t *>(a.y) + off64) = packed;
        }
    }
}

typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt with only the vector-memory count constrained (<= N outstanding)
template <int N>
__device__ __forceinline__ void wait_vmcnt_le()
{
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    // gfx9 encoding: vmcnt [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// VEC: X rows are 16-byte aligned and k % 16 == 0, so token rows are copied
// to LDS with 16-byte direct loads; otherwise they are staged byte by byte.
template <int KIND, int ST, int CT, int WM, int WN, int D, bool VEC>
__device__ __forceinline__ void sparse_linear_body(const LinearArgs &a, const GeluArg *ep)
{
    using S = Shape<ST, CT, WM, WN, D>;
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];

    const int64_t work = xcd_work_index(blockIdx.x, gridDim.x);
    const int64_t mt = work / a.n_cgroups;
    const int32_t cg = (int32_t)(work % a.n_cgroups);
    const int64_t m0 = mt * S::TM;
    const int32_t tile0 = cg * S::NT;
    const int32_t ntl = min(S::NT, a.n_tiles - tile0);
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int wm = wave % WM, wn = wave / WM;
    const size_t pstride = (size_t)a.n_tiles + 1;

    // per window: bit j set if tile tile0 + j has an overflow operand, and the
    // index of the workgroup's first overflow operand of the window
    uint2 *om = reinterpret_cast<uint2 *>(smem + S::LDS);
    for (int w = tid; w < a.n_win; w += S::NTH) {
        const uint32_t *p = a.ovf_ptr + (size_t)w * pstride + tile0;
        uint32_t mask = 0;
        for (int j = 0; j < ntl; ++j) mask |= (p[j + 1] > p[j] ? 1u : 0u) << j;
        om[w] = make_uint2(mask, p[0]);
    }
    GeluCell *tab = reinterpret_cast<GeluCell *>(smem + S::LDS + ((a.n_win * 8 + 15) & ~15));
    float hinv = 0.0f, eoff = 0.0f, cmax = 0.0f;
    if constexpr (KIND == SL_EPI_I8_GELU) {
        for (int u = tid; u < ep->nc; u += S::NTH) tab[u] = ep->cell[u];
        hinv = ep->hinv;
        eoff = ep->off;
        cmax = (float)(ep->nc - 1);
    }

    i32x4 acc[CT][ST];
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
        for (int s = 0; s < ST; ++s) acc[c][s] = i32x4{0, 0, 0, 0};

    // Copy sources, window-independent parts, per copy of this lane. A lane
    // without data copies valid bytes into padding: copies whose products are
    // never stored (rows past m) or meet zero weights (columns past k), or
    // operand slots no wave reads.
    const int8_t *xsrc[S::CX];
    int32_t xlim[S::CX];
#pragma unroll
    for (int i = 0; i < S::CX; ++i) {
        const int pc = (i * S::NW + wave) * 64 + lane;
        const int r = min(pc / kXRowPieces, S::TM - 1), pp = min(pc % kXRowPieces, kXRowPieces - 2);
        xsrc[i] = a.x + min(m0 + r, a.m - 1) * a.k + pp * 16;
        xlim[i] = a.k - 16 - pp * 16;
    }
    int32_t apiece[S::CA];
#pragma unroll
    for (int i = 0; i < S::CA; ++i) apiece[i] = (i * S::NW + wave) * 64 + lane;
    const int8_t *main0 = a.main + (size_t)tile0 * kOpBytes;

    // start window w's copies into buffer slot (global -> LDS, asynchronous)
    // o: the window's overflow mask entry, read by the caller
    auto issue = [&](int w, int slot, uint2 o) {
        int8_t *b = smem + slot * S::BUF;
        if (w >= a.n_win) w = a.n_win - 1;  // past the end: harmless repeat keeps the copy count fixed
        const uint32_t olo = __builtin_amdgcn_readfirstlane(o.y);
        const int nov = __builtin_popcount(__builtin_amdgcn_readfirstlane(o.x));
        // (without VEC the X rows are staged below and every step waits for
        // all copies, so the copy count need not be fixed)
        if constexpr (VEC) {
#pragma unroll
            for (int i = 0; i < S::CX; ++i) {
                const int p0 = (i * S::NW + wave) * 64;
                __builtin_amdgcn_global_load_lds(xsrc[i] + min(w * kWin, xlim[i]), (lds_void *)(b + p0 * 16), 16, 0,
                                                 0);
            }
        }
        const int8_t *mw = main0 + (size_t)w * a.n_tiles * kOpBytes;
#pragma unroll
        for (int i = 0; i < S::CA; ++i) {
            const int p0 = S::XP + (i * S::NW + wave) * 64;
            const int8_t *src = apiece[i] < ntl * kOpPieces ? mw + apiece[i] * 16 : a.main;
            __builtin_amdgcn_global_load_lds(src, (lds_void *)(b + p0 * 16), 16, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < S::CA; ++i) {
            const int p0 = S::XP + S::AP + (i * S::NW + wave) * 64;
            const int8_t *src =
                apiece[i] < nov * kOpPieces ? a.ovf + ((size_t)olo * kOpPieces + apiece[i]) * 16 : a.ovf;
            __builtin_amdgcn_global_load_lds(src, (lds_void *)(b + p0 * 16), 16, 0, 0);
        }
        if constexpr (!VEC) {
            for (int u = tid; u < S::TM * kWin; u += S::NTH) {
                const int r = u / kWin, c = u % kWin;
                const int64_t tok = m0 + r;
                const int32_t col = w * kWin + c;
                b[r * kXs + c] = (tok < a.m && col < a.k) ? a.x[tok * a.k + col] : (int8_t)0;
            }
        }
    };

    // this lane's B row offset (token) and 32-column slice of the window
    const int brow = (wm * ST * 16 + (lane & 15)) * kXs + 32 * (lane >> 4);
    // this lane's index word: block-row (lane%16)/4, lane group lane/16
    const int iword = ((lane & 15) >> 2) * 4 + (lane >> 4);

    auto step = [&](int w, int slot) {
        // window w (slot) has landed for this wave once at most D-2 later
        // windows' copies are outstanding; the barrier makes all waves' visible
        if constexpr (VEC)
            wait_vmcnt_le<(D - 2) * S::COPIES>();
        else
            __builtin_amdgcn_s_waitcnt(0);
        // a bare barrier: __syncthreads() would also wait for the later
        // windows' copies still in flight. The loop writes LDS only through
        // those counted copies; the clobber keeps the compiler from moving
        // LDS reads across the barrier.
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        const int8_t *b = smem + slot * S::BUF;
        i32x8 bv[ST];
#pragma unroll
        for (int s = 0; s < ST; ++s) {
            const int8_t *p = b + brow + s * 16 * kXs;
            const i32x4 lo = *reinterpret_cast<const i32x4 *>(p);
            const i32x4 hi = *reinterpret_cast<const i32x4 *>(p + 16);
            bv[s] = i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        }
        const uint32_t mask = __builtin_amdgcn_readfirstlane(om[w].x);
        // read here, with this window's reads, rather than after the first
        // copies of the step: the compiler drains all copies before an LDS
        // read it cannot separate from them
        const int wn1 = min(w + D - 1, a.n_win - 1);
        const uint2 onext = make_uint2(om[wn1].x, om[wn1].y);
        i32x4 av[CT], ao[CT];
        int ix[CT], io[CT];
#pragma unroll
        for (int c = 0; c < CT; ++c) {
            const int jw = wn * CT + c;
            const int8_t *op = b + S::XP * 16 + jw * kOpBytes;
            av[c] = *reinterpret_cast<const i32x4 *>(op + lane * 16);
            ix[c] = *reinterpret_cast<const int *>(op + 1024 + iword * 4);
            const int slot1 = __builtin_popcount(mask & ((1u << jw) - 1u));
            const int8_t *oo = b + (S::XP + S::AP) * 16 + slot1 * kOpBytes;
            ao[c] = *reinterpret_cast<const i32x4 *>(oo + lane * 16);
            io[c] = *reinterpret_cast<const int *>(oo + 1024 + iword * 4);
        }
        // the buffer read in the previous step is free: refill it
        issue(w + D - 1, (slot + D - 1) % D, onext);
#pragma unroll
        for (int c = 0; c < CT; ++c) {
            const int jw = wn * CT + c;
            if (jw < ntl) {
#pragma unroll
                for (int s = 0; s < ST; ++s)
                    acc[c][s] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(av[c], bv[s], acc[c][s], ix[c], 0, 0);
                if ((mask >> jw) & 1u) {
#pragma unroll
                    for (int s = 0; s < ST; ++s)
                        acc[c][s] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(ao[c], bv[s], acc[c][s], io[c], 0, 0);
                }
            }
        }
    };

    __syncthreads();  // overflow masks and epilogue table visible
    uint2 o0[D - 1];
#pragma unroll
    for (int d = 0; d < D - 1; ++d) o0[d] = make_uint2(om[min(d, a.n_win - 1)].x, om[min(d, a.n_win - 1)].y);
#pragma unroll
    for (int d = 0; d < D - 1; ++d) issue(d, d, o0[d]);
    int w = 0;
    for (; w + D <= a.n_win; w += D) {
#pragma unroll
        for (int u = 0; u < D; ++u) step(w + u, u);
    }
#pragma unroll
    for (int u = 0; u < D; ++u)
        if (w + u < a.n_win) step(w + u, u);
    __builtin_amdgcn_s_waitcnt(0);  // no copy may land after the workgroup ends

    // accumulator layout: lane l holds rows 4*(l/16)+r (channels of one
    // block-row), column l%16 (token), r = 0..3
#pragma unroll
    for (int c = 0; c < CT; ++c) {
        const int32_t t = tile0 + wn * CT + c;
        if (t >= a.n_tiles) break;
        const int32_t ch0 = t * kTileN + 4 * (lane >> 4);
        if (ch0 >= a.n) continue;  // block-rows past n_out in the last tile
        float s[4] = {0, 0, 0, 0}, bb4[4] = {0, 0, 0, 0};
        if constexpr (KIND != SL_EPI_ACC_I32) {
            const float4 sw = *reinterpret_cast<const float4 *>(a.w_scale + ch0);
            const float4 bb = *reinterpret_cast<const float4 *>(a.bias + ch0);
            s[0] = a.sx * sw.x;
            s[1] = a.sx * sw.y;
            s[2] = a.sx * sw.z;
            s[3] = a.sx * sw.w;
            bb4[0] = bb.x;
            bb4[1] = bb.y;
            bb4[2] = bb.z;
            bb4[3] = bb.w;
        }
#pragma unroll
        for (int st = 0; st < ST; ++st)
            epilogue_store<KIND>(a, acc[c][st], m0 + wm * ST * 16 + st * 16 + (lane & 15), ch0, s, bb4, tab, hinv,
                                 eoff, cmax);
    }
}

template <int KIND, int ST, int CT, int WM, int WN, int D, bool VEC>
__global__ __launch_bounds__(64 * WM * WN) void sparse_linear_kernel(LinearArgs a)
{
    sparse_linear_body<KIND, ST, CT, WM, WN, D, VEC>(a, nullptr);
}

template <int ST, int CT, int WM, int WN, int D, bool VEC>
__global__ __launch_bounds__(64 * WM * WN) void sparse_linear_gelu_kernel(LinearArgs a, GeluArg ep)
{
    sparse_linear_body<SL_EPI_I8_GELU, ST, CT, WM, WN, D, VEC>(a, &ep);
}

// ---------------------------------------------------------------------------
// activation quantisation

__device__ __forceinline__ uint32_t quant4(float4 v, float inv)
{
    return ((uint32_t)requant_i8(v.x, inv) & 0xffu) | (((uint32_t)requant_i8(v.y, inv) & 0xffu) << 8) |
           (((uint32_t)requant_i8(v.z, inv) & 0xffu) << 16) | (((uint32_t)requant_i8(v.w, inv) & 0xffu) << 24);
}

// 16 elements per thread per iteration: 4 x 16-byte loads, one 16-byte store.
__global__ __launch_bounds__(256) void quantize_vec16_kernel(const float *x, int64_t n16, float inv, int8_t *q)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) {
        const float4 *src = reinterpret_cast<const float4 *>(x) + 4 * i;
        uint4 o;
        o.x = quant4(src[0], inv);
        o.y = quant4(src[1], inv);
        o.z = quant4(src[2], inv);
        o.w = quant4(src[3], inv);
        reinterpret_cast<uint4 *>(q)[i] = o;
    }
}

__global__ __launch_bounds__(256) void quantize_scalar_kernel(const float *x, int64_t n, float inv, int8_t *q)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        q[i] = (int8_t)requant_i8(x[i], inv);
}

// ---------------------------------------------------------------------------
// host side

sl_status check_device_arch(int *device)
{
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    hipDeviceProp_t prop;
    HIP_TRY(hipGetDeviceProperties(&prop, dev));
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0) {
        set_error(std::string("device ") + std::to_string(dev) + " is " + prop.gcnArchName +
                  "; this library has gfx950 kernels only");
        return SL_ERR_UNSUPPORTED;
    }
    *device = dev;
    return SL_OK;
}

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

sl_status upload_image(sl_packed_weight *w)
{
    const TileImage &ti = w->tiles;
    const size_t b_main = std::max<size_t>(ti.main.size(), 16);
    const size_t b_ovf = std::max<size_t>(ti.ovf.size(), 16);
    const size_t b_ptr = ti.ovf_ptr.size() * sizeof(uint32_t);
    const size_t b_vec = (size_t)w->n_out * sizeof(float);
    const size_t o_main = 0;
    const size_t o_ovf = align256(o_main + b_main);
    const size_t o_ptr = align256(o_ovf + b_ovf);
    const size_t o_sw = align256(o_ptr + b_ptr);
    const size_t o_b = align256(o_sw + b_vec);
    const size_t total = align256(o_b + b_vec);
    void *base = nullptr;
    hipError_t e = hipMalloc(&base, total);
    if (e != hipSuccess) {
        set_error(std::string("hipMalloc of the packed weight: ") + hipGetErrorString(e));
        return e == hipErrorOutOfMemory ? SL_ERR_OOM : SL_ERR_HIP;
    }
    char *p = static_cast<char *>(base);
    w->dev.base = base;
    w->dev.bytes = (int64_t)total;
    w->on_device = true;  // from here on sparse_linear_free releases the memory
    if (!ti.main.empty()) HIP_TRY(hipMemcpy(p + o_main, ti.main.data(), ti.main.size(), hipMemcpyHostToDevice));
    if (!ti.ovf.empty()) HIP_TRY(hipMemcpy(p + o_ovf, ti.ovf.data(), ti.ovf.size(), hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p + o_ptr, ti.ovf_ptr.data(), b_ptr, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p + o_sw, w->w_scale.data(), b_vec, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p + o_b, w->bias.data(), b_vec, hipMemcpyHostToDevice));
    w->dev.main = reinterpret_cast<const int8_t *>(p + o_main);
    w->dev.ovf = reinterpret_cast<const int8_t *>(p + o_ovf);
    w->dev.ovf_ptr = reinterpret_cast<const uint32_t *>(p + o_ptr);
    w->dev.w_scale = reinterpret_cast<const float *>(p + o_sw);
    w->dev.bias = reinterpret_cast<const float *>(p + o_b);
    return SL_OK;
}

void release_image(sl_packed_weight *w)
{
    if (!w->dev.base) return;
    int cur = -1;
    const bool have_cur = hipGetDevice(&cur) == hipSuccess;
    if (w->dev.device >= 0) (void)hipSetDevice(w->dev.device);
    (void)hipDeviceSynchronize();
    (void)hipFree(w->dev.base);
    if (have_cur) (void)hipSetDevice(cur);
    w->dev.base = nullptr;
    w->on_device = false;
}

// Workgroup shapes (ST, CT, WM, WN, D): (16*ST*WM) tokens x (16*CT*WN)
// channels, D windows in flight.
struct TileCfg {
    int st, ct, wm, wn, d;
    int tm() const { return 16 * st * wm; }
    int nt() const { return ct * wn; }
};
static const TileCfg kCfgs[] = {
    {2, 3, 4, 2, 3},  // 128 x  96, 8 waves
    {2, 2, 2, 2, 4},  //  64 x  64, 4 waves
    {1, 2, 2, 2, 4},  //  32 x  64, 4 waves
    {1, 1, 2, 2, 4},  //  32 x  32, 4 waves
};

template <int KIND, int ST, int CT, int WM, int WN, int D, bool VEC>
static sl_status launch_cfg(const LinearArgs &a, const GeluArg *ep, int64_t nwg, hipStream_t stream)
{
    using S = Shape<ST, CT, WM, WN, D>;
    const void *fn;
    if constexpr (KIND == SL_EPI_I8_GELU)
        fn = reinterpret_cast<const void *>(&sparse_linear_gelu_kernel<ST, CT, WM, WN, D, VEC>);
    else
        fn = reinterpret_cast<const void *>(&sparse_linear_kernel<KIND, ST, CT, WM, WN, D, VEC>);
    static bool attr_done = false;  // benign race: setting it twice is harmless
    if (!attr_done) {
        HIP_TRY(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, kLdsMax));
        attr_done = true;
    }
    const size_t lds = (size_t)S::LDS + (((size_t)a.n_win * 8 + 15) & ~(size_t)15) +
                       (KIND == SL_EPI_I8_GELU ? kGeluCells * sizeof(GeluCell) : 0);
    if (lds > kLdsMax) {
        set_error("k_in too large for this workgroup shape's per-window table");
        return SL_ERR_UNSUPPORTED;
    }
    if constexpr (KIND == SL_EPI_I8_GELU)
        hipLaunchKernelGGL((sparse_linear_gelu_kernel<ST, CT, WM, WN, D, VEC>), dim3((uint32_t)nwg), dim3(S::NTH),
                           lds, stream, a, *ep);
    else
        hipLaunchKernelGGL((sparse_linear_kernel<KIND, ST, CT, WM, WN, D, VEC>), dim3((uint32_t)nwg), dim3(S::NTH),
                           lds, stream, a);
    HIP_TRY(hipGetLastError());
    return SL_OK;
}

template <int KIND, bool VEC>
static sl_status launch_kind(const LinearArgs &a, const GeluArg *ep, TileCfg c, int64_t nwg, hipStream_t stream)
{
#define SL_CFG(A_, B_, C_, D_, E_)                                                 \
    if (c.st == A_ && c.ct == B_ && c.wm == C_ && c.wn == D_ && c.d == E_) \
        return launch_cfg<KIND, A_, B_, C_, D_, E_, VEC>(a, ep, nwg, stream);
    SL_CFG(2, 3, 4, 2, 3)
    SL_CFG(2, 2, 2, 2, 4)
    SL_CFG(1, 2, 2, 2, 4)
#undef SL_CFG
    return launch_cfg<KIND, 1, 1, 2, 2, 4, VEC>(a, ep, nwg, stream);
}

template <int KIND>
static sl_status launch_vec(const LinearArgs &a, const GeluArg *ep, TileCfg c, int64_t nwg, hipStream_t stream,
                            bool vec)
{
    return vec ? launch_kind<KIND, true>(a, ep, c, nwg, stream) : launch_kind<KIND, false>(a, ep, c, nwg, stream);
}

// Pick the workgroup shape: among shapes that give every CU a workgroup,
// the one with the least L2 traffic (token rows re-read once per channel
// group, the weight image once per token group); SL_TILE="st,ct,wm,wn"
// overrides (tuning; unknown shapes are ignored).
static TileCfg choose_cfg(int64_t m, const sl_packed_weight *w)
{
    static const char *env = getenv("SL_TILE");
    if (env) {
        TileCfg c;
        if (sscanf(env, "%d,%d,%d,%d", &c.st, &c.ct, &c.wm, &c.wn) == 4)
            for (const TileCfg &k : kCfgs)
                if (k.st == c.st && k.ct == c.ct && k.wm == c.wm && k.wn == c.wn) return k;
    }
    const int32_t n_tiles = w->tiles.n_tiles;
    const double xbytes = (double)m * w->k_in;
    const double wbytes = (double)w->tiles.main.size() + (double)w->tiles.ovf.size();
    const TileCfg *best = nullptr, *most = nullptr;
    double best_cost = 0;
    int64_t most_wg = 0;
    for (const TileCfg &c : kCfgs) {
        const int64_t mt = (m + c.tm() - 1) / c.tm();
        const int64_t cgs = (n_tiles + c.nt() - 1) / c.nt();
        const int64_t nwg = mt * cgs;
        if (nwg > most_wg) {
            most_wg = nwg;
            most = &c;
        }
        if (nwg < 240) continue;
        const double cost = xbytes * cgs + wbytes * mt;
        if (!best || cost < best_cost) {
            best = &c;
            best_cost = cost;
        }
    }
    return best ? *best : *most;
}

sl_status launch_linear(const sl_packed_weight *w, const int8_t *x, int64_t m, float sx, int32_t kind,
                        float inv_so, void *y, void *stream)
{
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    if (dev != w->dev.device) {
        set_error("handle was packed on device " + std::to_string(w->dev.device) + ", current device is " +
                  std::to_string(dev));
        return SL_ERR_INVALID_ARG;
    }
    const TileImage &ti = w->tiles;
    LinearArgs a;
    a.x = x;
    a.y = y;
    a.m = m;
    a.n = w->n_out;
    a.k = w->k_in;
    a.main = w->dev.main;
    a.ovf = w->dev.ovf;
    a.ovf_ptr = w->dev.ovf_ptr;
    a.w_scale = w->dev.w_scale;
    a.bias = w->dev.bias;
    a.sx = sx;
    a.inv_so = inv_so;
    a.n_tiles = ti.n_tiles;
    a.n_win = ti.n_win;
    const bool vec = (w->k_in % 16 == 0) && ((reinterpret_cast<uintptr_t>(x) & 15) == 0);
    const TileCfg cfg = choose_cfg(m, w);
    a.n_cgroups = (ti.n_tiles + cfg.nt() - 1) / cfg.nt();
    const int64_t mt = (m + cfg.tm() - 1) / cfg.tm();
    const int64_t nwg = mt * a.n_cgroups;
    if (nwg > 0x7fffffff) {
        set_error("m_tokens too large for one launch");
        return SL_ERR_UNSUPPORTED;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    switch (kind) {
    case SL_EPI_ACC_I32: return launch_vec<SL_EPI_ACC_I32>(a, nullptr, cfg, nwg, s, vec);
    case SL_EPI_F32: return launch_vec<SL_EPI_F32>(a, nullptr, cfg, nwg, s, vec);
    case SL_EPI_F32_GELU: return launch_vec<SL_EPI_F32_GELU>(a, nullptr, cfg, nwg, s, vec);
    case SL_EPI_I8: return launch_vec<SL_EPI_I8>(a, nullptr, cfg, nwg, s, vec);
    default: {
        std::shared_ptr<const GeluTable> tab = gelu_table(inv_so);
        if (!tab->ok) return launch_vec<kEpiI8GeluErf>(a, nullptr, cfg, nwg, s, vec);
        GeluArg ga;
        ga.hinv = tab->hinv;
        ga.off = tab->off;
        ga.nc = tab->nc;
        ga.pad = 0;
        memcpy(ga.cell, tab->cell, sizeof(ga.cell));
        return launch_vec<SL_EPI_I8_GELU>(a, &ga, cfg, nwg, s, vec);
    }
    }
}

sl_status launch_quantize(const float *x, int64_t n, float inv_scale, int8_t *q, void *stream)
{
    hipStream_t s = static_cast<hipStream_t>(stream);
    const bool aligned = ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(q)) & 15) == 0;
    const int64_t n16 = aligned ? n / 16 : 0;
    if (n16 > 0) {
        const int64_t blocks = std::min<int64_t>((n16 + 255) / 256, 256 * 16);
        hipLaunchKernelGGL(quantize_vec16_kernel, dim3((uint32_t)blocks), dim3(256), 0, s, x, n16, inv_scale, q);
        HIP_TRY(hipGetLastError());
    }
    const int64_t rest = n - n16 * 16;
    if (rest > 0) {
        const int64_t blocks = std::min<int64_t>((rest + 255) / 256, 256 * 16);
        hipLaunchKernelGGL(quantize_scalar_kernel, dim3((uint32_t)blocks), dim3(256), 0, s, x + n16 * 16, rest,
                           inv_scale, q + n16 * 16);
        HIP_TRY(hipGetLastError());
    }
    return SL_OK;
}

}  // namespace sl
