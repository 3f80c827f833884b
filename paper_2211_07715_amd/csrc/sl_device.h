// Device-side definitions shared by the kernels of the sparse INT8 linear
// library (gfx950): launch arguments, the epilogue, wait helpers and the
// work-item iterator of the persistent workgroups. Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "sl_internal.h"

namespace sl {

typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

// Output store marked non-temporal: a kernel's outputs are read by a later
// kernel, never by itself, so they need not displace its inputs in the caches.
template <class V>
__device__ __forceinline__ void store_nt(void *p, V v)
{
    if constexpr (sizeof(V) == 4) {
        __builtin_nontemporal_store(__builtin_bit_cast(uint32_t, v), reinterpret_cast<uint32_t *>(p));
    } else if constexpr (sizeof(V) == 8) {
        __builtin_nontemporal_store(__builtin_bit_cast(i32x2, v), reinterpret_cast<i32x2 *>(p));
    } else {
        static_assert(sizeof(V) == 16, "4, 8 or 16-byte stores");
        __builtin_nontemporal_store(__builtin_bit_cast(i32x4, v), reinterpret_cast<i32x4 *>(p));
    }
}

constexpr int kXcds = 8;  // accelerator complex dies, each with its own L2
constexpr int kMaxDevices = 64;
// Buffer-load offset past any buffer this library reads (all < 2 GiB): such
// a lane reads zeros. Buffer word 3 for raw byte loads on gfx9.
constexpr uint32_t kOob = 0x80000000u;
constexpr int32_t kRsrcWord3 = 0x00020000;
constexpr int64_t kMaxBufferBytes = 0x7ff00000;  // per launch: token chunk bytes and weight image
constexpr int kVecLds = 512;  // a compute wave's weight scales and biases (staged kernel)
constexpr int kGeluLds = (kGeluCells * (int)sizeof(GeluCell) + 15) / 16 * 16;
constexpr int kMaskLds = 256;  // the ring buffers' overflow masks
constexpr size_t kLdsMax = 160 * 1024; // LDS per workgroup on gfx950

#define HIP_TRY(expr)                                                                     \
    do {                                                                                  \
        hipError_t e_ = (expr);                                                           \
        if (e_ != hipSuccess) {                                                           \
            set_error("%s: %s", #expr, hipGetErrorString(e_));                              \
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
    const int8_t *ovf;    // compact overflow operands (staged, weight-stationary kernels) or the dense
                          // overflow image (split-reduction, direct kernels)
    uint32_t main_bytes;  // image sizes: the range of the buffer loads
    uint32_t ovf_bytes;
    const uint32_t *om;  // overflow table of this launch's tile-group size, [n_win][n_cgroups][2]
    const float *w_scale;
    const float *bias;
    float sx;
    float inv_so;
    int32_t n_tiles;
    int32_t n_win;
    int32_t n_cgroups;  // channel groups of NT tiles
    int64_t n_items;    // work items: token tiles x channel groups
    int32_t x_cb;       // 32-feature column blocks of x (SL_LAYOUT_T16X32 input)
    int32_t y_cb;       // 32-channel column blocks of y (SL_LAYOUT_T16X32 output)
    // weight-stationary kernel only
    const int8_t *pan;      // panel image of this launch's channel-group size: per group, its window
                            // table ([n_win + 1][4] words) and panel, pan_instr KiB apart
    uint32_t pan_bytes;     // bytes of that image (the range of the copies)
    int32_t pan_instr;      // 1024-byte copies per channel group
    int32_t n_slices;       // token slices per channel group
    int32_t slice_groups;   // token groups (16 ST tokens) per slice
    // split-reduction kernel only: waves per workgroup
    int32_t kw;
};

// Byte offset of element (t, c) of an int8 tensor in SL_LAYOUT_T16X32 with
// cb column blocks: 512-byte blocks of 16 tokens x 32 features.
__device__ __forceinline__ int64_t t16x32_offset(int64_t t, int32_t c, int32_t cb)
{
    return ((t >> 4) * cb + (c >> 5)) * 512 + (t & 15) * 32 + (c & 31);
}

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

// Value stored for one accumulator group (4 channels of one token): int32
// accumulators, fp32 outputs, or 4 packed int8 codes.
template <int KIND>
struct EpiOut {
    using T = uint32_t;
    static constexpr int kBytes = 1;  // per channel
};
template <>
struct EpiOut<SL_EPI_ACC_I32> {
    using T = i32x4;
    static constexpr int kBytes = 4;
};
template <>
struct EpiOut<SL_EPI_F32> {
    using T = float4;
    static constexpr int kBytes = 4;
};
template <>
struct EpiOut<SL_EPI_F32_GELU> {
    using T = float4;
    static constexpr int kBytes = 4;
};

// 8-byte LDS read at a 32-bit LDS address
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u32x2 lds_read_u2(uint32_t addr)
{
    return *(const __attribute__((address_space(3))) u32x2 *)(uintptr_t)addr;
}

// The int8 GELU step-table epilogue in two halves, so that a caller can
// issue the table reads of many accumulator groups before it needs any:
// gelu_cells computes y = acc s + b (two fp32 roundings, as the definition)
// and the LDS address of y's cell for 4 accumulators; gelu_codes packs the
// 4 codes once the cells (threshold, then the two codes) have been read.
__device__ __forceinline__ void gelu_cells(const i32x4 acc, const float s[4], const float b[4], const GeluCell *tab,
                                           float hinv, float off, float cmax, float (&y)[4], uint32_t (&ad)[4])
{
#pragma clang fp contract(off)
    // (read through readfirstlane: a uniform register operand of the
    // shift-and-add, not a constant folded into two instructions)
    const uint32_t tab_adj = (uint32_t)__builtin_amdgcn_readfirstlane(
        (int)((uint32_t)(uintptr_t)(const __attribute__((address_space(3))) GeluCell *)tab -
              (__float_as_uint(kGeluBase) << 3)));
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float v = (float)acc[r] * s[r];
        v = v + b[r];
        y[r] = v;
        // the bits of c are those of kGeluBase plus the cell index (see
        // kGeluBase), so one shift-and-add with tab_adj = (LDS address of
        // the table) - 8 * bits(kGeluBase), modulo 2^32, gives the cell's
        // address
        const float c = __builtin_amdgcn_fmed3f(__builtin_fmaf(v, hinv, off), kGeluBase, cmax);
        ad[r] = (__float_as_uint(c) << 3) + tab_adj;
    }
}
__device__ __forceinline__ uint32_t gelu_codes(const float (&y)[4], const u32x2 (&cell)[4])
{
    // byte selectors of the permute that writes code r into byte r of the
    // packed word: earlier bytes kept (4 + i), byte r taken from the cell's
    // codes (0: q_lo, 1: q_hi), later bytes zero (0x0c)
    constexpr uint32_t kSelLo[4] = {0x0c0c0c00u, 0x0c0c0004u, 0x0c000504u, 0x00060504u};
    constexpr uint32_t kSelHi[4] = {0x0c0c0c01u, 0x0c0c0104u, 0x0c010504u, 0x01060504u};
    uint32_t packed = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r)
        packed = __builtin_amdgcn_perm(packed, cell[r].y, y[r] >= __uint_as_float(cell[r].x) ? kSelHi[r] : kSelLo[r]);
    return packed;
}

// Epilogue of one accumulator group: s = input scale x weight scales, b =
// biases of the 4 channels; tab, hinv, off, cmax (= kGeluBase + cells - 1):
// the GELU step table.
template <int KIND>
__device__ __forceinline__ typename EpiOut<KIND>::T epilogue_value_s(float inv_so, const i32x4 acc,
                                                                     const float s[4], const float b[4],
                                                                     const GeluCell *tab, float hinv, float off,
                                                                     float cmax)
{
#pragma clang fp contract(off)
    if constexpr (KIND == SL_EPI_ACC_I32) {
        return acc;
    } else if constexpr (KIND == SL_EPI_I8_GELU) {
        float y[4];
        uint32_t ad[4];
        gelu_cells(acc, s, b, tab, hinv, off, cmax, y, ad);
        u32x2 cell[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) cell[r] = lds_read_u2(ad[r]);
        return gelu_codes(y, cell);
    } else {
        float g[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float y = (float)acc[r] * s[r];
            y = y + b[r];
            g[r] = (KIND == SL_EPI_F32_GELU || KIND == kEpiI8GeluErf) ? gelu_erf(y) : y;
        }
        if constexpr (KIND == SL_EPI_F32 || KIND == SL_EPI_F32_GELU) {
            return make_float4(g[0], g[1], g[2], g[3]);
        } else {
            uint32_t packed = 0;
#pragma unroll
            for (int r = 0; r < 4; ++r) packed |= ((uint32_t)requant_i8(g[r], inv_so) & 0xffu) << (8 * r);
            return packed;
        }
    }
}

template <int KIND>
__device__ __forceinline__ typename EpiOut<KIND>::T epilogue_value(const LinearArgs &a, const i32x4 acc,
                                                                   const float s[4], const float b[4],
                                                                   const GeluCell *tab, float hinv, float off,
                                                                   float cmax)
{
    return epilogue_value_s<KIND>(a.inv_so, acc, s, b, tab, hinv, off, cmax);
}

// Epilogue and store of one accumulator group at token tok, channels
// ch0..ch0+3 (nothing past the last token). YT: y in SL_LAYOUT_T16X32 (int8
// kinds only), else row-major.
template <int KIND, bool YT = false>
__device__ __forceinline__ void epilogue_store(const LinearArgs &a, const i32x4 acc, int64_t tok, int32_t ch0,
                                               const float s[4], const float b[4], const GeluCell *tab,
                                               float hinv, float off, float cmax)
{
    if (tok >= a.m) return;
    static_assert(!YT || EpiOut<KIND>::kBytes == 1, "the block layout holds int8 outputs");
    const int64_t o = YT ? t16x32_offset(tok, ch0, a.y_cb) : (tok * a.n + ch0) * EpiOut<KIND>::kBytes;
    store_nt(static_cast<int8_t *>(a.y) + o, epilogue_value<KIND>(a, acc, s, b, tab, hinv, off, cmax));
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

// s_waitcnt with only the LDS / scalar-memory count constrained (none outstanding)
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4)); }

// Copy waves, start of step w: wait until element w+1 has landed. The copies
// issued after element w+1's last copy may stay outstanding: in the prologue
// order (token rows, main operands and overflow mask of elements 0..D-1, then
// their overflow operands) that is the overflow copies of elements w+2..D-1
// plus the elements copied in steps 0..w-1, later the D-2 elements copied
// after it.
template <int D, int CA, int COPIES, int I = 0>
__device__ __forceinline__ void wait_window_landed(int w)
{
    if constexpr (I < D - 2) {
        if (w == I) {
            wait_vmcnt_le<(D - 2 - I) * CA + I * COPIES>();
            return;
        }
        wait_window_landed<D, CA, COPIES, I + 1>(w);
    } else {
        wait_vmcnt_le<(D - 2) * COPIES>();
    }
}

// The work items of one workgroup: slot, slot + G, slot + 2G, ... as token
// tile mt, channel group cg and window rotation rot (items walk the windows
// from different starting points; integer accumulation does not depend on
// the order, and the workgroups that share an input or weight line then
// fetch it at different times). next() advances by G without dividing.
struct ItemIter {
    int32_t mt, cg, rot;
    int32_t dmt, dcg, drot;
    int32_t n_cgroups, n_win;
    __device__ static ItemIter start(int32_t slot, int32_t g, int32_t n_cgroups, int32_t n_win)
    {
        ItemIter it;
        it.mt = slot / n_cgroups;
        it.cg = slot - it.mt * n_cgroups;
        it.rot = (int32_t)(((int64_t)slot * 7) % n_win);
        it.dmt = g / n_cgroups;
        it.dcg = g - it.dmt * n_cgroups;
        it.drot = (int32_t)(((int64_t)g * 7) % n_win);
        it.n_cgroups = n_cgroups;
        it.n_win = n_win;
        return it;
    }
    __device__ void next()
    {
        mt += dmt;
        cg += dcg;
        if (cg >= n_cgroups) {
            cg -= n_cgroups;
            ++mt;
        }
        rot += drot;
        if (rot >= n_win) rot -= n_win;
    }
};

// Workgroup shapes of the direct-operand kernel (kernels_direct.hip): WM
// compute waves of ST 16-token subtiles x NT 16-channel tiles, D windows in
// flight. Only for 16-byte aligned token rows (k_in % 16 == 0).
struct DirectCfg {
    int st, nt, wm, d;
    int tm() const { return 16 * st * wm; }
};
constexpr int kNumDirectCfgs = 3;
extern const DirectCfg kDirectCfgs[kNumDirectCfgs];
// run_kind: an SL_EPI_* kind or kEpiI8GeluErf; ep: the GELU table for
// SL_EPI_I8_GELU; xt / yt: x / y in SL_LAYOUT_T16X32 (yt for int8 kinds)
sl_status launch_direct(const LinearArgs &a, const GeluArg *ep, int32_t run_kind, DirectCfg c, bool xt, bool yt,
                        hipStream_t stream);

// Split-reduction kernel (kernels_split.hip): one work item of kSplitSt
// 16-token subtiles x kSplitNt 16-channel tiles per workgroup of a.kw waves
// (1 <= kw <= kSplitMaxWaves), whose waves split the item's windows, at most
// split_windows_per_wave(n_win) each (1 or 2: the fewer that lets
// kSplitMaxWaves waves cover the windows; 0: too many windows, over 32, for
// this kernel). For few tokens; aligned or block-layout token rows.
constexpr int kSplitSt = 1;
constexpr int kSplitNt = 2;
constexpr int kSplitWin = 2;
constexpr int kSplitMaxWaves = 16;
constexpr int64_t kSplitAutoItems = 1280;  // automatic choice up to this many work items
int split_windows_per_wave(int32_t n_win);
sl_status launch_split(const LinearArgs &a, const GeluArg *ep, int32_t run_kind, bool xt, bool yt,
                       hipStream_t stream);

// Workgroup shapes of the weight-stationary kernel (kernels_panel.hip): NWV
// waves, each multiplying ST 16-token subtiles by the NT 16-channel tiles of
// the workgroup's channel group, whose whole weight panel sits in LDS; R
// windows of token rows in each wave's registers.
struct PanelCfg {
    int nt, st, nwv, r;
    int tg() const { return 16 * st; }
};
constexpr int kNumPanelCfgs = 5;
extern const PanelCfg kPanelCfgs[kNumPanelCfgs];
// LDS bytes of a panel kernel launch whose channel groups' tables and panels
// take `stride` bytes each
size_t panel_lds_bytes(PanelCfg c, int32_t run_kind, bool yt, uint32_t stride);
sl_status launch_panel(const LinearArgs &a, const GeluArg *ep, int32_t run_kind, PanelCfg c, bool xt, bool yt,
                       size_t lds, hipStream_t stream);
// resident workgroups of a panel-kernel shape for `lds` bytes of LDS (all kinds and layouts of a
// shape share one register budget; the SL_EPI_F32 row-major instance stands for them)
sl_status panel_resident(PanelCfg c, size_t lds, int *out);

// Persistent grid size of a kernel on the current device: the workgroups of
// `threads` threads and `lds` bytes of dynamic LDS resident at once. On first
// use per device it also raises the kernel's dynamic-LDS limit; cache holds
// kMaxDevices entries per kernel instance.
sl_status persistent_grid(const void *fn, int threads, size_t lds, int *cache, int *out);

}  // namespace sl
