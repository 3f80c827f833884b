// The split-reduction kernel of the sparse INT8 linear layer (gfx950): for
// few tokens (a batch of one sequence), where one workgroup per output tile
// walking the whole reduction would leave most of the chip idle and put
// every window's memory latency in series.
//
// Same method and operand image as the other kernels (Section "Sparse GEMM
// operators", Figure 1, Algorithm 1: the stored 4x1 blocks are one operand of
// the 4:2-sparse int8 matrix instruction, the input columns the weight's mask
// names are selected by the instruction's column indices, int32 accumulation,
// one fused epilogue per output). A workgroup owns one work item (ST 16-token
// subtiles x NT 16-channel tiles) and splits its reduction over its waves:
// wave v of kw takes windows v, v + kw, ... (at most WPW of them). It
// issues every load of its windows at once -- token rows, main and overflow
// operands, the latter from an overflow image laid out like the main one
// (one slot per window and tile, zeros where the tile has none, so that no
// lookup stands between a wave and its loads) -- and so waits about one
// memory latency before its matrix instructions. The waves' int32 partial sums meet in
// LDS; integer addition is exact in any order, so the sum equals the single
// accumulation of the other kernels bit for bit. Each (tile, subtile) pair
// is then reduced, and its epilogue run, by one wave.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "sl_device.h"

namespace sl {

// XT: x in SL_LAYOUT_T16X32 (else row-major, 16-byte aligned rows); YT: y in
// SL_LAYOUT_T16X32 (int8 kinds). The workgroup has a.kw waves of at most
// WPW windows each (a.kw * WPW >= n_win).
template <int KIND, int ST, int NT, int WPW, bool XT, bool YT>
__device__ __forceinline__ void split_body(const LinearArgs &a, const GeluArg *ep)
{
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int kw = a.kw;  // = blockDim.x / 64

    // channel-group-major items: the token tiles of one channel group run
    // on one XCD, which then fetches that group's weight operands once
    // (n_items < 2^31)
    const uint32_t item = (uint32_t)xcd_work_index(blockIdx.x, gridDim.x);
    const uint32_t n_mt = (uint32_t)((a.m + 16 * ST - 1) / (16 * ST));
    const int32_t cg = (int32_t)(item / n_mt);
    const int64_t t0 = (int64_t)(item - (uint32_t)cg * n_mt) * (16 * ST);
    const int32_t tile0 = cg * NT;
    const int32_t ntl = min(NT, a.n_tiles - tile0);

    // LDS: the partial sums ([kw][NT*ST] accumulator groups of 64 lanes),
    // then the GELU table
    i32x4 *part = reinterpret_cast<i32x4 *>(smem);
    GeluCell *tab = reinterpret_cast<GeluCell *>(smem + kw * NT * ST * 1024);
    // this wave's windows: w_j = wave + j * kw, j < nw
    const int nw = wave < a.n_win ? (a.n_win - 1 - wave) / kw + 1 : 0;

    const __amdgpu_buffer_rsrc_t mr = __builtin_amdgcn_make_buffer_rsrc((void *)a.main, 0, (int)a.main_bytes,
                                                                        kRsrcWord3);
    // (a.ovf: the overflow image in the main image's layout)
    const __amdgpu_buffer_rsrc_t orc = __builtin_amdgcn_make_buffer_rsrc((void *)a.ovf, 0, (int)a.ovf_bytes,
                                                                         kRsrcWord3);
    const int64_t xbytes = XT ? (a.m + 15) / 16 * a.x_cb * 512 : a.m * a.k;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.x, 0, (int)min<int64_t>(xbytes, kMaxBufferBytes), kRsrcWord3);
    const uint32_t wstride = (uint32_t)a.n_tiles * kOpBytes;  // main image bytes per window
    // this lane's index word: block-row (lane%16)/4, lane group lane/16
    const int iword = ((lane & 15) >> 2) * 4 + (lane >> 4);

    // Token rows: lane l of subtile s loads features 32*(l/16) .. +31 of
    // the window for token (l % 16) -- the B operand layout (as in the
    // direct kernel; tokens past m read zeros or a padding token of the last
    // block, a ragged last window bytes that meet zero weights).
    uint32_t ro[ST];
#pragma unroll
    for (int s = 0; s < ST; ++s) {
        const int64_t r = t0 + s * 16 + (lane & 15);
        if constexpr (XT)
            ro[s] = r < (a.m + 15) / 16 * 16 ? (uint32_t)((r >> 4) * a.x_cb * 512) + 512u * (uint32_t)(lane >> 4) +
                                                   32u * (uint32_t)(lane & 15)
                                             : kOob;
        else
            ro[s] = r < a.m ? (uint32_t)(r * a.k) + 32u * (uint32_t)(lane >> 4) : kOob;
    }

    i32x8 bv[WPW][ST];
    i32x4 av[WPW][NT], ao[WPW][NT];
    int ix[WPW][NT], io[WPW][NT];
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
        if (j < nw) {
            const uint32_t w = (uint32_t)(wave + j * kw);
#pragma unroll
            for (int s = 0; s < ST; ++s) {
                const uint32_t off = ro[s] + w * (XT ? 4 * 512 : kWin);
                const i32x4 lo = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
                const i32x4 hi =
                    __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off + 16u, 0, 0));
                bv[j][s] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            }
#pragma unroll
            for (int c = 0; c < NT; ++c) {
                const uint32_t base = c < ntl ? (uint32_t)(tile0 + c) * (uint32_t)kOpBytes : kOob;
                av[j][c] = __builtin_bit_cast(
                    i32x4, __builtin_amdgcn_raw_buffer_load_b128(mr, base + 16u * (uint32_t)lane, w * wstride, 0));
                ix[j][c] = (int)__builtin_amdgcn_raw_buffer_load_b32(mr, base + 1024u + 4u * (uint32_t)iword,
                                                                     w * wstride, 0);
                ao[j][c] = __builtin_bit_cast(
                    i32x4, __builtin_amdgcn_raw_buffer_load_b128(orc, base + 16u * (uint32_t)lane, w * wstride, 0));
                io[j][c] = (int)__builtin_amdgcn_raw_buffer_load_b32(orc, base + 1024u + 4u * (uint32_t)iword,
                                                                     w * wstride, 0);
            }
        }
    }

    // While those loads are in flight: the epilogue's weight scales and
    // biases of this wave's first (tile, subtile) pair (pair p = (tile c,
    // subtile s) goes to wave p % kw: a workgroup may have fewer waves than
    // pairs), and the GELU step table into LDS.
    auto load_vec = [&](int p, i32x4 &sw, i32x4 &b4) {
        const int32_t ch0 = (tile0 + p / ST) * kTileN + 4 * (lane >> 4);
        const __amdgpu_buffer_rsrc_t sr = __builtin_amdgcn_make_buffer_rsrc((void *)a.w_scale, 0, a.n * 4, kRsrcWord3);
        const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc((void *)a.bias, 0, a.n * 4, kRsrcWord3);
        const uint32_t off = ch0 < a.n ? (uint32_t)ch0 * 4u : kOob;
        sw = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(sr, off, 0, 0));
        b4 = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(br, off, 0, 0));
    };
    i32x4 sw0 = {0, 0, 0, 0}, b40 = {0, 0, 0, 0};
    if constexpr (KIND != SL_EPI_ACC_I32)
        if (wave < NT * ST) load_vec(wave, sw0, b40);
    float hinv = 0.0f, eoff = 0.0f, cmax = 0.0f;
    if constexpr (KIND == SL_EPI_I8_GELU) {
        for (int u = tid; u < ep->nc; u += (int)blockDim.x) tab[u] = ep->cell[u];
        hinv = ep->hinv;
        eoff = ep->off;
        cmax = kGeluBase + (float)(ep->nc - 1);
    }

    i32x4 acc[NT][ST];
#pragma unroll
    for (int c = 0; c < NT; ++c)
#pragma unroll
        for (int s = 0; s < ST; ++s) acc[c][s] = i32x4{0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < WPW; ++j) {
        if (j < nw) {
#pragma unroll
            for (int c = 0; c < NT; ++c)
#pragma unroll
                for (int s = 0; s < ST; ++s)
                    acc[c][s] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(av[j][c], bv[j][s], acc[c][s], ix[j][c], 0, 0);
#pragma unroll
            for (int c = 0; c < NT; ++c)
#pragma unroll
                for (int s = 0; s < ST; ++s)
                    acc[c][s] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(ao[j][c], bv[j][s], acc[c][s], io[j][c], 0, 0);
        }
    }
#pragma unroll
    for (int c = 0; c < NT; ++c)
#pragma unroll
        for (int s = 0; s < ST; ++s) part[((wave * NT + c) * ST + s) * 64 + lane] = acc[c][s];
    __syncthreads();

    // accumulator layout: lane l holds rows 4*(l/16)+r (channels of one
    // block-row), column l%16 (token), r = 0..3
    for (int p = wave; p < NT * ST; p += kw) {
        const int c = p / ST, s = p % ST;
        if (c < ntl) {
            i32x4 sum = part[(c * ST + s) * 64 + lane];
            for (int v = 1; v < kw; ++v) sum += part[((v * NT + c) * ST + s) * 64 + lane];
            const int32_t ch0 = (tile0 + c) * kTileN + 4 * (lane >> 4);
            const int64_t tok = t0 + s * 16 + (lane & 15);
            float sc[4] = {0.0f, 0.0f, 0.0f, 0.0f}, bb[4] = {0.0f, 0.0f, 0.0f, 0.0f};
            if constexpr (KIND != SL_EPI_ACC_I32) {
                i32x4 sw = sw0, b4 = b40;
                if (p != wave) load_vec(p, sw, b4);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    sc[r] = a.sx * __int_as_float(sw[r]);
                    bb[r] = __int_as_float(b4[r]);
                }
            }
            if (ch0 < a.n) epilogue_store<KIND, YT>(a, sum, tok, ch0, sc, bb, tab, hinv, eoff, cmax);
        }
    }
}

template <int KIND, int ST, int NT, int WPW, bool XT, bool YT>
__global__ __launch_bounds__(64 * kSplitMaxWaves) void sparse_linear_split_kernel(LinearArgs a)
{
    split_body<KIND, ST, NT, WPW, XT, YT>(a, nullptr);
}

template <int ST, int NT, int WPW, bool XT, bool YT>
__global__ __launch_bounds__(64 * kSplitMaxWaves) void sparse_linear_split_gelu_kernel(LinearArgs a, GeluArg ep)
{
    split_body<SL_EPI_I8_GELU, ST, NT, WPW, XT, YT>(a, &ep);
}

template <int KIND, int WPW, bool XT, bool YT>
static sl_status launch_split_wpw(const LinearArgs &a, const GeluArg *ep, hipStream_t stream)
{
    constexpr int ST = kSplitSt, NT = kSplitNt;
    const size_t lds = (size_t)a.kw * NT * ST * 1024 + (KIND == SL_EPI_I8_GELU ? kGeluLds : 0);
    const dim3 grid((uint32_t)a.n_items), block((uint32_t)(64 * a.kw));
    if constexpr (KIND == SL_EPI_I8_GELU)
        hipLaunchKernelGGL((sparse_linear_split_gelu_kernel<ST, NT, WPW, XT, YT>), grid, block, lds, stream, a, *ep);
    else
        hipLaunchKernelGGL((sparse_linear_split_kernel<KIND, ST, NT, WPW, XT, YT>), grid, block, lds, stream, a);
    HIP_TRY(hipGetLastError());
    return SL_OK;
}

template <int KIND, bool XT, bool YT>
static sl_status launch_split_kind(const LinearArgs &a, const GeluArg *ep, int wpw, hipStream_t stream)
{
    static_assert(kSplitWin == 2, "one instance per windows-per-wave count");
    if (wpw == 1) return launch_split_wpw<KIND, 1, XT, YT>(a, ep, stream);
    return launch_split_wpw<KIND, 2, XT, YT>(a, ep, stream);
}

template <int KIND, bool XT>
static sl_status launch_split_y(const LinearArgs &a, const GeluArg *ep, int wpw, bool yt, hipStream_t stream)
{
    if constexpr (EpiOut<KIND>::kBytes == 1)
        if (yt) return launch_split_kind<KIND, XT, true>(a, ep, wpw, stream);
    return launch_split_kind<KIND, XT, false>(a, ep, wpw, stream);
}

template <int KIND>
static sl_status launch_split_x(const LinearArgs &a, const GeluArg *ep, int wpw, bool xt, bool yt,
                                hipStream_t stream)
{
    return xt ? launch_split_y<KIND, true>(a, ep, wpw, yt, stream) : launch_split_y<KIND, false>(a, ep, wpw, yt, stream);
}

int split_windows_per_wave(int32_t n_win)
{
    for (int wpw = 1; wpw <= kSplitWin; wpw *= 2)
        if (n_win <= wpw * kSplitMaxWaves) return wpw;
    return 0;
}

sl_status launch_split(const LinearArgs &a, const GeluArg *ep, int32_t run_kind, bool xt, bool yt,
                       hipStream_t stream)
{
    const int wpw = split_windows_per_wave(a.n_win);
    if (wpw == 0 || a.kw < 1 || a.kw > kSplitMaxWaves || (int64_t)a.kw * wpw < a.n_win ||
        a.n_items > 0x7fffffff) {
        set_error("internal: split-reduction launch out of range");
        return SL_ERR_UNSUPPORTED;
    }
    if (a.n_items == 0) return SL_OK;
    switch (run_kind) {
    case SL_EPI_ACC_I32: return launch_split_x<SL_EPI_ACC_I32>(a, nullptr, wpw, xt, yt, stream);
    case SL_EPI_F32: return launch_split_x<SL_EPI_F32>(a, nullptr, wpw, xt, yt, stream);
    case SL_EPI_F32_GELU: return launch_split_x<SL_EPI_F32_GELU>(a, nullptr, wpw, xt, yt, stream);
    case SL_EPI_I8: return launch_split_x<SL_EPI_I8>(a, nullptr, wpw, xt, yt, stream);
    case SL_EPI_I8_GELU: return launch_split_x<SL_EPI_I8_GELU>(a, ep, wpw, xt, yt, stream);
    default: return launch_split_x<kEpiI8GeluErf>(a, nullptr, wpw, xt, yt, stream);
    }
}

}  // namespace sl
