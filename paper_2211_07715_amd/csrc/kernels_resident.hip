// The register-resident kernel of the sparse INT8 linear layer (gfx950).
//
// Same method as the other kernels (Section "Sparse GEMM operators", Figure 1,
// Algorithm 1): every stored 4x1 block is a value of the A operand of the
// 4:2-sparse int8 matrix instruction v_smfmac_i32_16x16x128_i8, whose 2-bit
// column indices select the input columns the block mask names; int32
// accumulation; one fused epilogue per output after the whole reduction.
//
// Schedule. A workgroup is 4 waves, one per SIMD. Each wave owns kResTiles
// 16-channel tiles and a slice of kResWin 128-column windows, and loads the
// main operands of those (tile, window) pairs into its registers once: the
// weights stay resident for the whole launch. The workgroup then walks its
// range of token passes (16 ST tokens each). The pass's token tile -- all K
// columns, in 512-byte blocks of 16 tokens x 32 columns -- is copied global to
// LDS (no registers) one pass ahead, double-buffered. Per window a wave reads
// its dense B operands from that tile and issues its tiles' matrix
// instructions: no weight traffic and almost no vector-ALU work in the loop.
// The rare third and fourth stored blocks of an aligned 4-column group sit in
// a few consolidated overflow operands per (tile, K slice), resident in LDS;
// their B operands are gathered from the token tile at 4-byte granularity,
// one column group per slot, at offsets the packer computed. When K spans
// more than one wave's slice, the waves of a channel part split the
// reduction and sum their int32 partials through LDS (exact in any order).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "sl_device.h"

namespace sl {

// Calls f(std::integral_constant<int, 0>) .. f(std::integral_constant<int, N-1>) in order.
template <int... Us, class F>
__device__ __forceinline__ void rs_for_impl(std::integer_sequence<int, Us...>, F &&f)
{
    (f(std::integral_constant<int, Us>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void rs_for(F &&f)
{
    rs_for_impl(std::make_integer_sequence<int, N>{}, f);
}

template <int KIND, int ST>
__global__ __launch_bounds__(kResThreads) __attribute__((amdgpu_waves_per_eu(1, 1))) void
sparse_linear_resident_kernel(ResArgs a, GeluArg ep)
{
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];
    constexpr int NT = kResTiles, NW = kResWin;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kp = wave % a.ks;  // K slice of this wave
    const int cp = wave / a.ks;  // channel part of this wave

    // work: token slice and channel group; the workgroups of one XCD take
    // consecutive works, which share a token slice
    const int32_t work = (int32_t)xcd_work_index(blockIdx.x, gridDim.x);
    const int32_t slice = work / a.n_cg;
    const int32_t cg = work - slice * a.n_cg;
    const int32_t p_begin = (int32_t)((int64_t)slice * a.passes / a.wg_per_cg);
    const int32_t p_end = (int32_t)((int64_t)(slice + 1) * a.passes / a.wg_per_cg);
    const int32_t tile_wg0 = cg * a.tiles_wg;
    const int32_t my_tile0 = tile_wg0 + cp * NT;
    const int32_t win0 = kp * NW;
    const int32_t nmw = std::max(0, std::min(NW, a.n_win - win0));

    const ResLds L = res_lds_layout(ST, a.cbw, a.tiles_wg, a.ks, KIND == SL_EPI_I8_GELU, a.lds_ovf);
    const float *const vec = reinterpret_cast<const float *>(smem + L.vec);

    // ---- token tile copies: pass p -> buffer b, in 1024-byte instructions;
    // instruction i covers column blocks 2i', 2i'+1 of subtile s, and lane L
    // copies piece L % 32 (token (L % 32) / 2, columns 16 (L % 2)) of the
    // block L / 32
    const int64_t xbytes = a.xt ? (a.m + 15) / 16 * a.x_cb * 512 : a.m * a.k;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.x, 0, (int)std::min<int64_t>(xbytes, kMaxBufferBytes), kRsrcWord3);
    const int half_cbw = a.cbw / 2;
    auto copy_x = [&](int32_t p, int b) {
        const int64_t t0 = (int64_t)p * 16 * ST;
        int8_t *const dst = smem + (uint32_t)b * L.xbuf;
        const int nins = ST * half_cbw;
        const int piece = lane & 31;
        for (int i = wave; i < nins; i += kResWaves) {
            const int s = i / half_cbw;
            const int cb = 2 * (i - s * half_cbw) + (lane >> 5);
            uint32_t off;
            if (a.xt) {
                // blocks past the tensor's columns (cb >= x_cb) read the next
                // blocks or zeros: they meet zero weights
                off = (uint32_t)((((t0 >> 4) + s) * a.x_cb + cb) * 512) + (uint32_t)piece * 16u;
            } else {
                // columns past k_in read the next row or zeros, likewise
                const int64_t tok = t0 + 16 * s + (piece >> 1);
                const int64_t col = (int64_t)cb * 32 + (piece & 1) * 16;
                off = tok < a.m ? (uint32_t)(tok * a.k + col) : kOob;
            }
            __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void *)(dst + (size_t)i * 1024), 16, off, 0, 0, 0);
        }
    };

    if (p_begin < p_end) copy_x(p_begin, 0);

    // ---- resident main operands: (my tile c, my window w); absent pairs
    // (past the last tile or window) read zeros and add nothing
    const __amdgpu_buffer_rsrc_t mr =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.main, 0, (int)a.main_bytes, kRsrcWord3);
    const uint32_t iword = (uint32_t)(((lane & 15) >> 2) * 4 + (lane >> 4));
    i32x4 av[NT][NW];
    int ix[NT][NW];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int c = 0; c < NT; ++c) {
            const bool ok = w < nmw && my_tile0 + c < a.n_tiles;
            const uint32_t off = ok ? (uint32_t)((win0 + w) * a.n_tiles + my_tile0 + c) * (uint32_t)kOpBytes : kOob;
            av[c][w] =
                __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(mr, off + (uint32_t)lane * 16u, 0, 0));
            ix[c][w] = __builtin_bit_cast(int, __builtin_amdgcn_raw_buffer_load_b32(mr, off + 1024u + iword * 4u, 0, 0));
        }

    // ---- the group's consolidated overflow operands, copied into LDS
    const int32_t tiles_end = std::min(tile_wg0 + a.tiles_wg, a.n_tiles);
    const uint32_t op_first = a.rdir[(size_t)tile_wg0 * a.ks];
    {
        const uint32_t op_last = a.rdir[(size_t)tiles_end * a.ks];
        const uint32_t nb = (op_last - op_first) * (uint32_t)kResOpBytes;
        const __amdgpu_buffer_rsrc_t orr =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.rovf, 0, (int)a.rovf_bytes, kRsrcWord3);
        const uint32_t src = op_first * (uint32_t)kResOpBytes + (uint32_t)lane * 16u;
        for (uint32_t i = (uint32_t)wave; i * 1024u < nb; i += kResWaves)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(orr, (lds_void *)(smem + L.ovf + i * 1024u), 16,
                                                     src + i * 1024u, 0, 0, 0);
    }
    // LDS byte range of my tiles' overflow operands in my K slice
    uint32_t ob[NT], oe[NT];
#pragma unroll
    for (int c = 0; c < NT; ++c) {
        const int32_t t = my_tile0 + c;
        if (t < a.n_tiles) {
            ob[c] = L.ovf + (a.rdir[(size_t)t * a.ks + kp] - op_first) * (uint32_t)kResOpBytes;
            oe[c] = L.ovf + (a.rdir[(size_t)t * a.ks + kp + 1] - op_first) * (uint32_t)kResOpBytes;
        } else {
            ob[c] = oe[c] = 0;
        }
    }

    // ---- set-up: per channel the dequantisation scale sx * sw[n] (one fp32
    // product, as in the definition) and the bias; the GELU step table
    if constexpr (KIND != SL_EPI_ACC_I32) {
        float *const vw = reinterpret_cast<float *>(smem + L.vec);
        for (int i = tid; i < a.tiles_wg * kTileN; i += kResThreads) {
            const int32_t ch = tile_wg0 * kTileN + i;
            vw[2 * i] = ch < a.n ? a.sx * a.w_scale[ch] : 0.0f;
            vw[2 * i + 1] = ch < a.n ? a.bias[ch] : 0.0f;
        }
    }
    float hinv = 0.0f, goff = 0.0f, cmax = 0.0f;
    if constexpr (KIND == SL_EPI_I8_GELU) {
        GeluCell *const tab = reinterpret_cast<GeluCell *>(smem + L.tab);
        for (int u = tid; u < ep.nc; u += kResThreads) tab[u] = ep.cell[u];
        hinv = ep.hinv;
        goff = ep.off;
        cmax = kGeluBase + (float)(ep.nc - 1);
    }
    wait_vmcnt_le<0>();
    __syncthreads();

    // ---- epilogue and store of one accumulator group: tile c of this wave's
    // channel part (0 .. NT-1), 16-token subtile from token tok0. A lane holds
    // the 4 channels 4 (lane / 16) .. +3 of the tile for token lane % 16.
    const int64_t mlim = a.yt ? (a.m + 15) / 16 * 16 : a.m;  // block layout: padding tokens may be written
    int8_t *const y8 = static_cast<int8_t *>(a.y);
    auto epilogue = [&](const i32x4 v, int c, int64_t tok0) {
        const int32_t tile = my_tile0 + c;
        const int32_t ch0 = tile * kTileN + 4 * (lane >> 4);
        const int64_t tok = tok0 + (lane & 15);
        if (tile >= a.n_tiles || ch0 >= a.n || tok >= mlim) return;
        if constexpr (KIND == SL_EPI_ACC_I32) {
            store_nt(y8 + (tok * a.n + ch0) * 4, v);
            return;
        } else {
            const int vi = (tile - tile_wg0) * kTileN + 4 * (lane >> 4);
            const float4 sb01 = *reinterpret_cast<const float4 *>(vec + 2 * vi);
            const float4 sb23 = *reinterpret_cast<const float4 *>(vec + 2 * vi + 4);
            const float s[4] = {sb01.x, sb01.z, sb23.x, sb23.z};
            const float b[4] = {sb01.y, sb01.w, sb23.y, sb23.w};
            if constexpr (KIND == SL_EPI_I8_GELU) {
#pragma clang fp contract(off)
                // GELU + requantisation by the step table: the cell is
                // med3(fma(y, hinv, off)) = kGeluBase (2^23) + index, whose
                // low 24 bits are the index; one 8-byte read gives the cell's
                // threshold and its two codes
                const int8_t *const tabp = smem + L.tab;
                uint32_t packed = 0;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float y = (float)v[r] * s[r];
                    y = y + b[r];
                    const float cf = __builtin_amdgcn_fmed3f(__builtin_fmaf(y, hinv, goff), kGeluBase, cmax);
                    const uint2 cell = *reinterpret_cast<const uint2 *>(tabp + __umul24(__float_as_uint(cf), 8u));
                    const uint32_t q = y >= __uint_as_float(cell.x) ? cell.y >> 8 : cell.y;
                    packed |= (q & 0xffu) << (8 * r);
                }
                const int64_t o = a.yt ? t16x32_offset(tok, ch0, a.y_cb) : tok * a.n + ch0;
                store_nt(y8 + o, packed);
            } else {
                const auto val = epilogue_value_s<KIND>(a.inv_so, v, s, b, nullptr, 0.0f, 0.0f, 0.0f);
                if constexpr (EpiOut<KIND>::kBytes == 1) {
                    const int64_t o = a.yt ? t16x32_offset(tok, ch0, a.y_cb) : tok * a.n + ch0;
                    store_nt(y8 + o, val);
                } else {
                    store_nt(y8 + (tok * a.n + ch0) * 4, val);
                }
            }
        }
    };

    // this lane's token row in a token-tile buffer, at window 0 of the wave's
    // slice: block (4 win0 + lane / 16), row lane % 16 (a wave whose slice
    // lies past k_in reads window 0: its weights are all zero)
    const uint32_t brow = (uint32_t)(4 * (nmw > 0 ? win0 : 0) + (lane >> 4)) * 512u + (uint32_t)(lane & 15) * 32u;
    const uint32_t sub_stride = (uint32_t)a.cbw * 512u;  // one 16-token subtile of the tile
    // reduction partners: groups g = c * ST + s of a channel part go to wave
    // kp' = g % ks of that part, which sums the ks partials
    int8_t *const red = smem + L.red;

    for (int32_t p = p_begin, it = 0; p < p_end; ++p, ++it) {
        const int buf = it & 1;
        // the other buffer was last read in the previous pass, which every
        // wave has finished (barrier at the end of it)
        const int64_t t0 = (int64_t)p * 16 * ST;
        const int8_t *const xb = smem + (uint32_t)buf * L.xbuf;
        i32x4 acc[NT][ST];
#pragma unroll
        for (int c = 0; c < NT; ++c)
#pragma unroll
            for (int s = 0; s < ST; ++s) acc[c][s] = i32x4{0, 0, 0, 0};

        // consolidated overflow operands: B gathered 4 bytes a slot
#pragma unroll
        for (int c = 0; c < NT; ++c) {
            for (uint32_t o = ob[c]; o < oe[c]; o += (uint32_t)kResOpBytes) {
                const int8_t *const op = smem + o;
                const i32x4 ao = *reinterpret_cast<const i32x4 *>(op + lane * 16);
                const int io = *reinterpret_cast<const int *>(op + 1024 + iword * 4);
                // slots 8 q .. 8 q + 7 of lane group q: offsets of their groups
                const uint4 g0 = *reinterpret_cast<const uint4 *>(op + kOpBytes + (lane >> 4) * 32);
                const uint4 g1 = *reinterpret_cast<const uint4 *>(op + kOpBytes + (lane >> 4) * 32 + 16);
                const uint32_t go[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
                const int8_t *const rb = xb + (uint32_t)(lane & 15) * 32u;
#pragma unroll
                for (int s = 0; s < ST; ++s) {
                    i32x8 bo;
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        bo[j] = *reinterpret_cast<const int *>(rb + go[j] + (uint32_t)s * sub_stride);
                    acc[c][s] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(ao, bo, acc[c][s], io, 0, 0);
                }
            }
        }

        if (p + 1 < p_end) copy_x(p + 1, buf ^ 1);
        // main windows: B of window w + 1 read while window w multiplies
        auto read_b = [&](i32x8 (&bv)[ST], int w) {
#pragma unroll
            for (int s = 0; s < ST; ++s) {
                const int8_t *const pb = xb + brow + (uint32_t)w * 2048u + (uint32_t)s * sub_stride;
                const i32x4 lo = *reinterpret_cast<const i32x4 *>(pb);
                const i32x4 hi = *reinterpret_cast<const i32x4 *>(pb + 16);
                bv[s] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            }
        };
        // (no branches: a window past the slice multiplies zero weights by the
        // slice's first window, which stays inside the tile)
        i32x8 bv[2][ST];
        read_b(bv[0], 0);
        rs_for<NW>([&](auto wc) {
            constexpr int W = decltype(wc)::value;
            if constexpr (W + 1 < NW) read_b(bv[(W + 1) & 1], W + 1 < nmw ? W + 1 : 0);
#pragma unroll
            for (int c = 0; c < NT; ++c)
#pragma unroll
                for (int s = 0; s < ST; ++s)
                    acc[c][s] =
                        __builtin_amdgcn_smfmac_i32_16x16x128_i8(av[c][W], bv[W & 1][s], acc[c][s], ix[c][W], 0, 0);
        });

        if (a.ks == 1) {
            // every wave has finished reading its token tile; its copies for
            // the next pass have landed before the epilogue's stores are issued
            // (so that the wait below does not wait for them)
            wait_vmcnt_le<0>();
#pragma unroll
            for (int c = 0; c < NT; ++c)
#pragma unroll
                for (int s = 0; s < ST; ++s) epilogue(acc[c][s], c, t0 + 16 * s);
        } else {
            // split reduction: partials to LDS, then wave kp of each part sums
            // the groups g with g % ks == kp
            int8_t *const mine = red + (uint32_t)wave * (NT * ST * 1024u);
#pragma unroll
            for (int c = 0; c < NT; ++c)
#pragma unroll
                for (int s = 0; s < ST; ++s)
                    *reinterpret_cast<i32x4 *>(mine + (c * ST + s) * 1024 + lane * 16) = acc[c][s];
            wait_vmcnt_le<0>();
            wait_lgkm0();  // LDS writes done
            __builtin_amdgcn_s_barrier();
            for (int g = kp; g < NT * ST; g += a.ks) {
                i32x4 sum = i32x4{0, 0, 0, 0};
                for (int k2 = 0; k2 < a.ks; ++k2)
                    sum += *reinterpret_cast<const i32x4 *>(red + (uint32_t)(cp * a.ks + k2) * (NT * ST * 1024u) +
                                                            (uint32_t)g * 1024u + (uint32_t)lane * 16u);
                epilogue(sum, g / ST, t0 + 16 * (g % ST));
            }
        }
        // the next pass reads the other buffer (copies waited for above, by
        // every wave) and overwrites this one: all waves are past this pass
        wait_lgkm0();
        __builtin_amdgcn_s_barrier();
    }
}

// ---------------------------------------------------------------------------
// host side

template <int KIND, int ST>
static sl_status launch_res_cfg(const ResArgs &a, const GeluArg *ep, uint32_t grid, size_t lds, hipStream_t stream)
{
    const void *fn = reinterpret_cast<const void *>(&sparse_linear_resident_kernel<KIND, ST>);
    static int raised[kMaxDevices] = {};  // per kernel instance and device: LDS limit raised
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) {
        set_error("device index beyond the supported range");
        return SL_ERR_UNSUPPORTED;
    }
    if (!raised[dev]) {
        HIP_TRY(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax));
        raised[dev] = 1;
    }
    static const GeluArg kNoTable{};
    hipLaunchKernelGGL((sparse_linear_resident_kernel<KIND, ST>), dim3(grid), dim3(kResThreads), lds, stream, a,
                       ep ? *ep : kNoTable);
    HIP_TRY(hipGetLastError());
    return SL_OK;
}

template <int ST>
static sl_status launch_res_st(const ResArgs &a, const GeluArg *ep, int32_t run_kind, uint32_t grid, size_t lds,
                               hipStream_t stream)
{
    switch (run_kind) {
    case SL_EPI_ACC_I32: return launch_res_cfg<SL_EPI_ACC_I32, ST>(a, nullptr, grid, lds, stream);
    case SL_EPI_F32: return launch_res_cfg<SL_EPI_F32, ST>(a, nullptr, grid, lds, stream);
    case SL_EPI_F32_GELU: return launch_res_cfg<SL_EPI_F32_GELU, ST>(a, nullptr, grid, lds, stream);
    case SL_EPI_I8: return launch_res_cfg<SL_EPI_I8, ST>(a, nullptr, grid, lds, stream);
    case SL_EPI_I8_GELU: return launch_res_cfg<SL_EPI_I8_GELU, ST>(a, ep, grid, lds, stream);
    default: return launch_res_cfg<kEpiI8GeluErf, ST>(a, nullptr, grid, lds, stream);
    }
}

sl_status launch_resident(const ResArgs &a, const GeluArg *ep, int32_t run_kind, int st, uint32_t grid, size_t lds,
                          hipStream_t stream)
{
    if (st == 1) return launch_res_st<1>(a, ep, run_kind, grid, lds, stream);
    set_error("internal: unknown register-resident subtile count");
    return SL_ERR_UNSUPPORTED;
}

}  // namespace sl
