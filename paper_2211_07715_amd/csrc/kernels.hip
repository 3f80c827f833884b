// gfx950 kernels of the sparse INT8 linear layer, and their launchers.
//
// Method (Section "Sparse GEMM operators", Figure 1, Algorithm 1): the stored
// 4x1 weight blocks form the A operand of an int8 dot-product instruction;
// the input columns named by the weight's mask are gathered ("re-organised")
// into the B operand; products accumulate in int32; bias and the other
// post-operators are applied once per output before the store.
//
// MI355X mapping used here:
//  * A workgroup (4 waves) owns a 64-token tile of X and a group of 16-channel
//    weight tiles. The token tile is staged once per k-chunk into LDS,
//    transposed to input-column-major order (one LDS row of 64 tokens per
//    input column), so a gather by column index reads whole LDS rows.
//  * Each wave owns some channel tiles. Per k-step it loads one 1 KiB A panel
//    (16 channels x 64 gathered positions, pre-laid-out by the packer in lane
//    order: one 16-byte load per lane, fully coalesced) and, for each of the 4
//    16-token subtiles, gathers the matching 16 x 64 int8 B block from LDS and
//    issues v_mfma_i32_16x16x64_i8 into that subtile's int32 accumulators.
//  * After the last k-chunk the epilogue (dequantise, bias, GELU(erf),
//    requantise) runs on the accumulators in registers and each lane stores 4
//    consecutive channels of one token.
#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include <algorithm>
#include <string>

#include "sl_internal.h"

namespace sl {

typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int kTM = 64;             // tokens per workgroup tile
constexpr int kSub = kTM / 16;      // 16-token subtiles per tile
constexpr int kWaves = 4;           // waves per workgroup
constexpr int kThreads = kWaves * 64;
constexpr int kLdsStride = kTM + 8; // bytes per staged input column (8-byte aligned rows)
constexpr int kXcds = 8;            // accelerator complex dies (each with its own L2)

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
    const uint32_t *seg_ptr;
    const int8_t *panel;
    const uint16_t *ucol;
    const float *w_scale;
    const float *bias;
    float sx;
    float inv_so;
    int32_t n_tiles;
    int32_t kc;
    int32_t n_chunks;
    int32_t tiles_per_group;
    int32_t n_groups;
    int32_t vec_stage;  // 1: X rows are 16-byte aligned and k % 16 == 0
};

// Workgroups are dispatched round-robin over the XCDs. Renumber them so that
// each XCD runs a contiguous range of work items (work items that share a
// token tile are adjacent, so that tile's X rows are fetched into one L2).
__device__ __forceinline__ int64_t xcd_work_index(int64_t bid, int64_t nwg)
{
    const int64_t q = nwg / kXcds, r = nwg % kXcds;
    const int64_t x = bid % kXcds, j = bid / kXcds;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

// 4x4 byte transpose: out[j] = {r0.byte j, r1.byte j, r2.byte j, r3.byte j}.
__device__ __forceinline__ void transpose4x4(uint32_t r0, uint32_t r1, uint32_t r2, uint32_t r3, uint32_t out[4])
{
    const uint32_t lo01 = __builtin_amdgcn_perm(r1, r0, 0x05010400u);
    const uint32_t hi01 = __builtin_amdgcn_perm(r1, r0, 0x07030602u);
    const uint32_t lo23 = __builtin_amdgcn_perm(r3, r2, 0x05010400u);
    const uint32_t hi23 = __builtin_amdgcn_perm(r3, r2, 0x07030602u);
    out[0] = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
    out[1] = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);
    out[2] = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
    out[3] = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);
}

// Stage X[m0 .. m0+63][kbeg .. kbeg+kw) into LDS as xt[kk][t] (row stride
// kLdsStride), zero for tokens >= m.
__device__ __forceinline__ void stage_tile(const LinearArgs &a, int64_t m0, int32_t kbeg, int32_t kw,
                                           uint8_t *lds)
{
    const int tid = threadIdx.x;
    if (a.vec_stage) {
        const int kg_n = kw / 16;
        const int units = (kTM / 4) * kg_n;
        for (int u = tid; u < units; u += kThreads) {
            const int kg = u % kg_n, tg = u / kg_n;
            uint4 r[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int64_t tok = m0 + tg * 4 + i;
                if (tok < a.m)
                    r[i] = *reinterpret_cast<const uint4 *>(a.x + tok * a.k + kbeg + kg * 16);
                else
                    r[i] = make_uint4(0, 0, 0, 0);
            }
            uint32_t o[4];
            uint8_t *dst = lds + (size_t)(kg * 16) * kLdsStride + tg * 4;
            transpose4x4(r[0].x, r[1].x, r[2].x, r[3].x, o);
#pragma unroll
            for (int j = 0; j < 4; ++j) *reinterpret_cast<uint32_t *>(dst + (0 + j) * kLdsStride) = o[j];
            transpose4x4(r[0].y, r[1].y, r[2].y, r[3].y, o);
#pragma unroll
            for (int j = 0; j < 4; ++j) *reinterpret_cast<uint32_t *>(dst + (4 + j) * kLdsStride) = o[j];
            transpose4x4(r[0].z, r[1].z, r[2].z, r[3].z, o);
#pragma unroll
            for (int j = 0; j < 4; ++j) *reinterpret_cast<uint32_t *>(dst + (8 + j) * kLdsStride) = o[j];
            transpose4x4(r[0].w, r[1].w, r[2].w, r[3].w, o);
#pragma unroll
            for (int j = 0; j < 4; ++j) *reinterpret_cast<uint32_t *>(dst + (12 + j) * kLdsStride) = o[j];
        }
    } else {
        const int total = kTM * kw;
        for (int i = tid; i < total; i += kThreads) {
            const int t = i / kw, kk = i % kw;
            const int64_t tok = m0 + t;
            lds[(size_t)kk * kLdsStride + t] = tok < a.m ? (uint8_t)a.x[tok * a.k + kbeg + kk] : (uint8_t)0;
        }
    }
}

// B operand for one 16-token subtile: lane l (token l%16 of the subtile, lane
// group l/16) receives the 16 input bytes at the gathered positions
// 16*(l/16) .. +15 of the k-step, i.e. at the columns cols[0..15].
__device__ __forceinline__ i32x4 gather_b(const uint8_t *lds, const uint16_t cols[16], int kbeg, int tok)
{
    uint32_t w[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        uint32_t v = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const uint32_t byte = lds[(size_t)(cols[4 * d + b] - kbeg) * kLdsStride + tok];
            v |= byte << (8 * b);
        }
        w[d] = v;
    }
    return i32x4{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
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
__device__ __forceinline__ void epilogue_store(const LinearArgs &a, const i32x4 acc, int64_t tok, int32_t ch0)
{
#pragma clang fp contract(off)
    if (tok >= a.m || ch0 >= a.n) return;
    const int64_t off = tok * a.n + ch0;
    if constexpr (KIND == SL_EPI_ACC_I32) {
        *reinterpret_cast<i32x4 *>(static_cast<int32_t *>(a.y) + off) = acc;
        return;
    } else {
        const float4 sw = *reinterpret_cast<const float4 *>(a.w_scale + ch0);
        const float4 bb = *reinterpret_cast<const float4 *>(a.bias + ch0);
        const float swv[4] = {sw.x, sw.y, sw.z, sw.w};
        const float bv[4] = {bb.x, bb.y, bb.z, bb.w};
        float g[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float s = a.sx * swv[r];
            float y = (float)acc[r] * s;
            y = y + bv[r];
            g[r] = (KIND == SL_EPI_F32_GELU || KIND == SL_EPI_I8_GELU) ? gelu_erf(y) : y;
        }
        if constexpr (KIND == SL_EPI_F32 || KIND == SL_EPI_F32_GELU) {
            *reinterpret_cast<float4 *>(static_cast<float *>(a.y) + off) = make_float4(g[0], g[1], g[2], g[3]);
        } else {
            uint32_t packed = 0;
#pragma unroll
            for (int r = 0; r < 4; ++r) packed |= ((uint32_t)requant_i8(g[r], a.inv_so) & 0xffu) << (8 * r);
            *reinterpret_cast<uint32_t *>(static_cast<int8_t *>(a.y) + off) = packed;
        }
    }
}

template <int KIND, int TW>
__global__ __launch_bounds__(kThreads) void sparse_linear_kernel(LinearArgs a)
{
    extern __shared__ __align__(16) uint8_t lds[];
    const int64_t work = xcd_work_index(blockIdx.x, gridDim.x);
    const int64_t tt = work / a.n_groups;
    const int32_t grp = (int32_t)(work % a.n_groups);
    const int64_t m0 = tt * kTM;
    const int32_t tile_begin = grp * a.tiles_per_group;
    const int32_t tile_end = min(a.n_tiles, tile_begin + a.tiles_per_group);
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;

    i32x4 acc[TW][kSub];
#pragma unroll
    for (int i = 0; i < TW; ++i)
#pragma unroll
        for (int s = 0; s < kSub; ++s) acc[i][s] = i32x4{0, 0, 0, 0};

    for (int32_t c = 0; c < a.n_chunks; ++c) {
        const int32_t kbeg = c * a.kc;
        const int32_t kw = min(a.k, kbeg + a.kc) - kbeg;
        __syncthreads();
        stage_tile(a, m0, kbeg, kw, lds);
        __syncthreads();
#pragma unroll
        for (int i = 0; i < TW; ++i) {
            const int32_t t = tile_begin + wave + i * kWaves;
            if (t >= tile_end) break;
            const uint32_t s0 = a.seg_ptr[(int64_t)t * a.n_chunks + c];
            const uint32_t s1 = a.seg_ptr[(int64_t)t * a.n_chunks + c + 1];
            for (uint32_t s = s0; s < s1; ++s) {
                const i32x4 av = *reinterpret_cast<const i32x4 *>(a.panel + (int64_t)s * kStepBytes + lane * 16);
                const uint16_t *uc = a.ucol + (int64_t)s * kStepK + (lane / 16) * 16;
                uint16_t cols[16];
                const uint4 c0 = *reinterpret_cast<const uint4 *>(uc);
                const uint4 c1 = *reinterpret_cast<const uint4 *>(uc + 8);
                memcpy(cols, &c0, 16);
                memcpy(cols + 8, &c1, 16);
#pragma unroll
                for (int sub = 0; sub < kSub; ++sub) {
                    const i32x4 bv = gather_b(lds, cols, kbeg, sub * 16 + lane % 16);
                    acc[i][sub] = __builtin_amdgcn_mfma_i32_16x16x64_i8(av, bv, acc[i][sub], 0, 0, 0);
                }
            }
        }
    }

    // accumulator lane layout of the 16x16 int32 result: lane l holds rows
    // 4*(l/16) + r (channels), column l%16 (token), r = 0..3
#pragma unroll
    for (int i = 0; i < TW; ++i) {
        const int32_t t = tile_begin + wave + i * kWaves;
        if (t >= tile_end) break;
        const int32_t ch0 = t * kTileN + 4 * (lane / 16);
#pragma unroll
        for (int sub = 0; sub < kSub; ++sub)
            epilogue_store<KIND>(a, acc[i][sub], m0 + sub * 16 + lane % 16, ch0);
    }
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
    const size_t b_seg = ti.seg_ptr.size() * sizeof(uint32_t);
    const size_t b_panel = ti.panel.size();
    const size_t b_ucol = ti.ucol.size() * sizeof(uint16_t);
    const size_t b_vec = (size_t)w->n_out * sizeof(float);
    const size_t o_seg = 0;
    const size_t o_panel = align256(o_seg + b_seg);
    const size_t o_ucol = align256(o_panel + b_panel);
    const size_t o_sw = align256(o_ucol + b_ucol);
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
    HIP_TRY(hipMemcpy(p + o_seg, ti.seg_ptr.data(), b_seg, hipMemcpyHostToDevice));
    if (b_panel) HIP_TRY(hipMemcpy(p + o_panel, ti.panel.data(), b_panel, hipMemcpyHostToDevice));
    if (b_ucol) HIP_TRY(hipMemcpy(p + o_ucol, ti.ucol.data(), b_ucol, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p + o_sw, w->w_scale.data(), b_vec, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p + o_b, w->bias.data(), b_vec, hipMemcpyHostToDevice));
    w->dev.seg_ptr = reinterpret_cast<const uint32_t *>(p + o_seg);
    w->dev.panel = reinterpret_cast<const int8_t *>(p + o_panel);
    w->dev.ucol = reinterpret_cast<const uint16_t *>(p + o_ucol);
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

template <int KIND, int TW>
static sl_status launch_kt(const LinearArgs &a, int64_t nwg, size_t lds_bytes, hipStream_t stream)
{
    static bool attr_done = false;  // benign race: setting the attribute twice is harmless
    if (!attr_done) {
        HIP_TRY(hipFuncSetAttribute(reinterpret_cast<const void *>(&sparse_linear_kernel<KIND, TW>),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, kChunkMax * kLdsStride));
        attr_done = true;
    }
    hipLaunchKernelGGL((sparse_linear_kernel<KIND, TW>), dim3((uint32_t)nwg), dim3(kThreads), lds_bytes, stream, a);
    HIP_TRY(hipGetLastError());
    return SL_OK;
}

template <int KIND>
static sl_status launch_kind(const LinearArgs &a, int tw, int64_t nwg, size_t lds_bytes, hipStream_t stream)
{
    switch (tw) {
    case 1: return launch_kt<KIND, 1>(a, nwg, lds_bytes, stream);
    case 2: return launch_kt<KIND, 2>(a, nwg, lds_bytes, stream);
    case 3: return launch_kt<KIND, 3>(a, nwg, lds_bytes, stream);
    default: return launch_kt<KIND, 4>(a, nwg, lds_bytes, stream);
    }
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
    a.seg_ptr = w->dev.seg_ptr;
    a.panel = w->dev.panel;
    a.ucol = w->dev.ucol;
    a.w_scale = w->dev.w_scale;
    a.bias = w->dev.bias;
    a.sx = sx;
    a.inv_so = inv_so;
    a.n_tiles = ti.n_tiles;
    a.kc = ti.kc;
    a.n_chunks = ti.n_chunks;
    a.vec_stage = (w->k_in % 16 == 0) && ((reinterpret_cast<uintptr_t>(x) & 15) == 0);

    const int64_t ntt = (m + kTM - 1) / kTM;
    // channel tiles per workgroup: as many as keep >= 2 workgroups per CU
    int tw = 1;
    for (int cand = 4; cand >= 1; --cand) {
        const int64_t groups = (ti.n_tiles + kWaves * cand - 1) / (kWaves * cand);
        if (ntt * groups >= 512) {
            tw = cand;
            break;
        }
    }
    a.tiles_per_group = kWaves * tw;
    a.n_groups = (ti.n_tiles + a.tiles_per_group - 1) / a.tiles_per_group;
    const int64_t nwg = ntt * a.n_groups;
    if (nwg > 0x7fffffff) {
        set_error("m_tokens too large for one launch");
        return SL_ERR_UNSUPPORTED;
    }
    const size_t lds_bytes = (size_t)ti.kc * kLdsStride;
    hipStream_t s = static_cast<hipStream_t>(stream);
    switch (kind) {
    case SL_EPI_ACC_I32: return launch_kind<SL_EPI_ACC_I32>(a, tw, nwg, lds_bytes, s);
    case SL_EPI_F32: return launch_kind<SL_EPI_F32>(a, tw, nwg, lds_bytes, s);
    case SL_EPI_F32_GELU: return launch_kind<SL_EPI_F32_GELU>(a, tw, nwg, lds_bytes, s);
    case SL_EPI_I8: return launch_kind<SL_EPI_I8>(a, tw, nwg, lds_bytes, s);
    default: return launch_kind<SL_EPI_I8_GELU>(a, tw, nwg, lds_bytes, s);
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
