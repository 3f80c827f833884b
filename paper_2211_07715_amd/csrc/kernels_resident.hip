// The register-resident kernel of the sparse INT8 linear layer (gfx950).
//
// Same method as the other kernels (Section "Sparse GEMM operators", Figure 1,
// Algorithm 1): every stored 4x1 block is a value of the A operand of the
// 4:2-sparse int8 matrix instruction v_smfmac_i32_16x16x128_i8, whose 2-bit
// column indices select the input columns the block mask names; int32
// accumulation; one fused epilogue per output after the whole reduction.
//
// Schedule. A workgroup is 4 compute waves, one per SIMD, and one memory
// wave. Each compute wave owns kResTiles 16-channel tiles and a slice of
// kResWin 128-column windows, and loads the main operands of those (tile,
// window) pairs into its registers once: the weights stay resident for the
// whole launch. The workgroup then walks its range of token passes of 16
// tokens. The memory wave copies each pass's token tile -- all K columns, in
// 512-byte blocks of 16 tokens x 32 columns -- global to LDS (no registers)
// one pass ahead into a second buffer, and writes the previous pass's outputs
// from an LDS staging buffer to memory, so the compute waves never touch
// global memory after the set-up and never wait for it. Per window a compute
// wave reads its dense B operands from the token tile and issues its tiles'
// matrix instructions: no weight traffic and almost no vector-ALU work in the
// loop. The rare third and fourth stored blocks of an aligned 4-column group
// sit in a few consolidated overflow operands per (tile, K slice), resident in
// LDS; their B operands are gathered from the token tile at 4-byte
// granularity, one column group per slot, at offsets the packer computed.
// When K spans more than one wave's slice, the compute waves of a channel
// part split the reduction and sum their int32 partials through LDS (exact
// in any order).
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

template <int KIND>
__global__ __launch_bounds__(kResThreads) __attribute__((amdgpu_waves_per_eu(1, 2))) void
sparse_linear_resident_kernel(ResArgs a, GeluArg ep)
{
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];
    constexpr int NT = kResTiles, NW = kResWin;
    constexpr int OB = EpiOut<KIND>::kBytes;  // output bytes per channel
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool mover = wave == kResWaves;

    // work: token slice and channel group; the workgroups of one XCD take
    // consecutive works, which share a token slice
    const int32_t work = (int32_t)xcd_work_index(blockIdx.x, gridDim.x);
    const int32_t slice = work / a.n_cg;
    const int32_t cg = work - slice * a.n_cg;
    const int32_t p_begin = (int32_t)((int64_t)slice * a.passes / a.wg_per_cg);
    const int32_t p_end = (int32_t)((int64_t)(slice + 1) * a.passes / a.wg_per_cg);
    const int32_t tile_wg0 = cg * a.tiles_wg;
    const int32_t tiles_end = std::min(tile_wg0 + a.tiles_wg, a.n_tiles);

    const ResLds L = res_lds_layout(a.cbw, a.tiles_wg, a.ks, OB, KIND == SL_EPI_I8_GELU, a.lds_ovf);
    const uint32_t op_first = a.rdir[(size_t)tile_wg0 * a.ks];

    // ---- set-up. The memory wave fills LDS: per channel the dequantisation
    // scale sx * sw[n] (one fp32 product, as in the definition) and the bias,
    // the GELU table, the index words of the group's main operands, the
    // all-zero overflow operand, the group's consolidated overflow operands
    // and the first token tile. The compute waves load their main operands;
    // the first pass waits for each window's operands as it reaches them.
    if (mover) {
        // =================== the memory wave ===================
        if constexpr (KIND != SL_EPI_ACC_I32) {
            float *const vw = reinterpret_cast<float *>(smem + L.vec);
            for (int i = lane; i < a.tiles_wg * kTileN; i += 64) {
                const int32_t ch = tile_wg0 * kTileN + i;
                vw[2 * i] = ch < a.n ? a.sx * a.w_scale[ch] : 0.0f;
                vw[2 * i + 1] = ch < a.n ? a.bias[ch] : 0.0f;
            }
        }
        if constexpr (KIND == SL_EPI_I8_GELU) {
            GeluCell *const tab = reinterpret_cast<GeluCell *>(smem + L.tab);
            for (int u = lane; u < ep.nc; u += 64) tab[u] = ep.cell[u];
        }
        for (int i = lane; i < kResOpBytes / 16; i += 64)
            *reinterpret_cast<uint4 *>(smem + L.dummy + i * 16) = uint4{0u, 0u, 0u, 0u};
        const __amdgpu_buffer_rsrc_t mr =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.main, 0, (int)a.main_bytes, kRsrcWord3);
        {
            // index words: (tile tl, window w) -> LDS (tl * n_win + w) * 64, four
            // lanes a pair, 16 pairs an instruction; tiles past the last read zeros
            const int32_t npairs = a.tiles_wg * a.n_win;
            for (int32_t i = 0; i * 16 < npairs; ++i) {
                const int32_t pr = i * 16 + (lane >> 2);
                const int32_t tl = pr / a.n_win, w = pr - tl * a.n_win;
                const uint32_t off = (pr < npairs && tile_wg0 + tl < a.n_tiles)
                                         ? (uint32_t)(w * a.n_tiles + tile_wg0 + tl) * (uint32_t)kOpBytes + 1024u +
                                               (uint32_t)(lane & 3) * 16u
                                         : kOob;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(mr, (lds_void *)(smem + L.idx + (uint32_t)i * 1024u), 16,
                                                         off, 0, 0, 0);
            }
        }
        {
            const uint32_t op_last = a.rdir[(size_t)tiles_end * a.ks];
            const uint32_t nb = (op_last - op_first) * (uint32_t)kResOpBytes;
            const __amdgpu_buffer_rsrc_t orr =
                __builtin_amdgcn_make_buffer_rsrc((void *)a.rovf, 0, (int)a.rovf_bytes, kRsrcWord3);
            const uint32_t src = op_first * (uint32_t)kResOpBytes + (uint32_t)lane * 16u;
            for (uint32_t i = 0; i * 1024u < nb; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(orr, (lds_void *)(smem + L.ovf + i * 1024u), 16,
                                                         src + i * 1024u, 0, 0, 0);
        }
        // token tile copies: pass p -> buffer b, 1024-byte instructions;
        // instruction i covers column blocks 2i, 2i+1, and lane L copies piece
        // L % 32 (token (L % 32) / 2, columns 16 (L % 2)) of block 2i + L / 32
        const int64_t xbytes = a.xt ? (a.m + 15) / 16 * a.x_cb * 512 : a.m * a.k;
        const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
            (void *)a.x, 0, (int)std::min<int64_t>(xbytes, kMaxBufferBytes), kRsrcWord3);
        const int piece = lane & 31;
        auto copy_x = [&](int32_t p, int b) {
            const int64_t t0 = (int64_t)p * 16;
            int8_t *const dst = smem + (uint32_t)b * L.xbuf;
            for (int i = 0; i < a.cbw / 2; ++i) {
                const int cb = 2 * i + (lane >> 5);
                uint32_t off;
                if (a.xt) {
                    // blocks past the tensor's columns (cb >= x_cb) read the
                    // next blocks or zeros: they meet zero weights
                    off = (uint32_t)(((t0 >> 4) * a.x_cb + cb) * 512) + (uint32_t)piece * 16u;
                } else {
                    // columns past k_in read the next row or zeros, likewise
                    const int64_t tok = t0 + (piece >> 1);
                    const int64_t col = (int64_t)cb * 32 + (piece & 1) * 16;
                    off = tok < a.m ? (uint32_t)(tok * a.k + col) : kOob;
                }
                __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void *)(dst + (size_t)i * 1024), 16, off, 0, 0, 0);
            }
        };
        // outputs of pass p from staging buffer b (16 token rows of the
        // group's channels) to y
        int8_t *const y8 = static_cast<int8_t *>(a.y);
        const int32_t row_pieces = a.tiles_wg * 4;  // 4-channel pieces of a row
        auto store_out = [&](int32_t p, int b) {
            const int8_t *const src = smem + L.out + (uint32_t)b * L.obuf;
            const int64_t t0 = (int64_t)p * 16;
            if (OB == 1 && a.yt) {
                // block layout: one tile's 16 channels of one token are 16
                // contiguous bytes of a 512-byte block (16 tokens x 32 channels)
                for (int i = lane; i < a.tiles_wg * 16; i += 64) {
                    const int32_t tl = i >> 4, t = i & 15;
                    const int32_t ch = (tile_wg0 + tl) * kTileN;
                    if (ch >= a.n) continue;
                    const uint4 v = *reinterpret_cast<const uint4 *>(src + (uint32_t)t * L.ostride + tl * kTileN);
                    store_nt(y8 + ((t0 >> 4) * a.y_cb + (ch >> 5)) * 512 + t * 32 + (ch & 31), v);
                }
            } else {
                for (int i = lane; i < 16 * row_pieces; i += 64) {
                    const int32_t t = i / row_pieces, q = i - t * row_pieces;
                    const int32_t ch = tile_wg0 * kTileN + 4 * q;
                    if (t0 + t >= a.m || ch >= a.n) continue;
                    const int8_t *const s = src + (uint32_t)t * L.ostride + (uint32_t)q * 4u * OB;
                    if constexpr (OB == 1)
                        store_nt(y8 + (t0 + t) * a.n + ch, *reinterpret_cast<const uint32_t *>(s));
                    else
                        store_nt(y8 + ((t0 + t) * a.n + ch) * 4, *reinterpret_cast<const uint4 *>(s));
                }
            }
        };
        if (p_begin < p_end) copy_x(p_begin, 0);
        wait_vmcnt_le<0>();
        wait_lgkm0();
        __builtin_amdgcn_s_barrier();
        for (int32_t p = p_begin, it = 0; p < p_end; ++p, ++it) {
            const int buf = it & 1;
            if (p + 1 < p_end) copy_x(p + 1, buf ^ 1);
            if (p > p_begin) store_out(p - 1, buf ^ 1);
            if (a.ks > 1) {
                // the compute waves' split reduction: two barriers
                __builtin_amdgcn_s_barrier();
                __builtin_amdgcn_s_barrier();
            }
            wait_vmcnt_le<0>();
            wait_lgkm0();
            __builtin_amdgcn_s_barrier();  // end of pass p
        }
        if (p_begin < p_end) store_out(p_end - 1, (p_end - 1 - p_begin) & 1);
        return;
    }

    // =================== the compute waves ===================
    const int kp = wave % a.ks;  // K slice of this wave
    const int cp = wave / a.ks;  // channel part of this wave
    const int32_t my_tile0 = tile_wg0 + cp * NT;
    const int32_t win0 = kp * NW;
    const int32_t nmw = std::max(0, std::min(NW, a.n_win - win0));
    const float *const vec = reinterpret_cast<const float *>(smem + L.vec);

    // resident main operands: (my tile c, my window w); absent pairs (past
    // the last tile or window) read zeros and add nothing. Issued window by
    // window, so the first pass can start on window 0 while the rest land.
    const __amdgpu_buffer_rsrc_t mr =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.main, 0, (int)a.main_bytes, kRsrcWord3);
    const uint32_t iword = (uint32_t)(((lane & 15) >> 2) * 4 + (lane >> 4));
    i32x4 av[NT][NW];
#pragma unroll
    for (int w = 0; w < NW; ++w)
#pragma unroll
        for (int c = 0; c < NT; ++c) {
            const bool ok = w < nmw && my_tile0 + c < a.n_tiles;
            const uint32_t off = ok ? (uint32_t)((win0 + w) * a.n_tiles + my_tile0 + c) * (uint32_t)kOpBytes : kOob;
            av[c][w] =
                __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(mr, off + (uint32_t)lane * 16u, 0, 0));
        }
    // LDS byte range of my tiles' overflow operands in my K slice, and the
    // first of them (the all-zero operand when a tile has none)
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
    float hinv = 0.0f, goff = 0.0f, cmax = 0.0f;
    if constexpr (KIND == SL_EPI_I8_GELU) {
        hinv = ep.hinv;
        goff = ep.off;
        cmax = kGeluBase + (float)(ep.nc - 1);
    }
    // (no wait for the main operands: only for what the memory wave put in LDS)
    __builtin_amdgcn_s_barrier();

    // index word of (my tile c, window w) for this lane
    const int8_t *const idxp = smem + L.idx + (uint32_t)((my_tile0 - tile_wg0) * a.n_win) * 64u + iword * 4u;
    const uint32_t idx_tile = (uint32_t)a.n_win * 64u;
    // this lane's token row in a token-tile buffer, at window 0 of the wave's
    // slice: block (4 win0 + lane / 16), row lane % 16 (a wave whose slice
    // lies past k_in reads window 0: its weights are all zero)
    const uint32_t wbase = (uint32_t)(nmw > 0 ? win0 : 0);
    const uint32_t brow = (uint32_t)(4 * wbase + (lane >> 4)) * 512u + (uint32_t)(lane & 15) * 32u;

    // epilogue of one accumulator group into the staging buffer: tile c of
    // this wave's channel part (0 .. NT-1); a lane holds the 4 channels
    // 4 (lane / 16) .. +3 of the tile for token row lane % 16
    auto epilogue = [&](const i32x4 v, int c, int8_t *obuf) {
        const int32_t tile = my_tile0 + c;
        if (tile >= a.n_tiles) return;
        const int cl = (tile - tile_wg0) * kTileN + 4 * (lane >> 4);  // channel within the group
        int8_t *const dst = obuf + (uint32_t)(lane & 15) * L.ostride + (uint32_t)cl * OB;
        if constexpr (KIND == SL_EPI_ACC_I32) {
            *reinterpret_cast<i32x4 *>(dst) = v;
        } else {
            const float4 sb01 = *reinterpret_cast<const float4 *>(vec + 2 * cl);
            const float4 sb23 = *reinterpret_cast<const float4 *>(vec + 2 * cl + 4);
            const float s[4] = {sb01.x, sb01.z, sb23.x, sb23.z};
            const float b[4] = {sb01.y, sb01.w, sb23.y, sb23.w};
            const auto val = epilogue_value_s<KIND>(a.inv_so, v, s, b, nullptr, 0.0f, 0.0f, 0.0f);
            *reinterpret_cast<typename EpiOut<KIND>::T *>(dst) = val;
        }
    };
    // The int8 GELU epilogue of all NT groups, two groups in flight: the step
    // table reads of group c are issued before group c - 1's codes are
    // formed. The cell is med3(fma(y, hinv, off)) = kGeluBase (2^23) + index,
    // whose low 24 bits are the index; one 8-byte read gives the cell's
    // threshold and its two codes.
    auto gelu_epilogue = [&](const i32x4 (&acc)[NT], int8_t *obuf) {
#pragma clang fp contract(off)
        const int8_t *const tabp = smem + L.tab;
        float y[2][4];
        uint2 cell[2][4];
        rs_for<NT + 1>([&](auto cc) {
            constexpr int C = decltype(cc)::value;
            if constexpr (C < NT) {
                const int cl = (my_tile0 + C - tile_wg0) * kTileN + 4 * (lane >> 4);
                const float4 sb01 = *reinterpret_cast<const float4 *>(vec + 2 * cl);
                const float4 sb23 = *reinterpret_cast<const float4 *>(vec + 2 * cl + 4);
                const float s[4] = {sb01.x, sb01.z, sb23.x, sb23.z};
                const float b[4] = {sb01.y, sb01.w, sb23.y, sb23.w};
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float yy = (float)acc[C][r] * s[r];
                    yy = yy + b[r];
                    y[C & 1][r] = yy;
                    const float cf = __builtin_amdgcn_fmed3f(__builtin_fmaf(yy, hinv, goff), kGeluBase, cmax);
                    cell[C & 1][r] = *reinterpret_cast<const uint2 *>(tabp + __umul24(__float_as_uint(cf), 8u));
                }
            }
            if constexpr (C > 0) {
                constexpr int P = C - 1;
                uint32_t packed = 0;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const uint32_t q = y[P & 1][r] >= __uint_as_float(cell[P & 1][r].x) ? cell[P & 1][r].y >> 8
                                                                                         : cell[P & 1][r].y;
                    packed |= (q & 0xffu) << (8 * r);
                }
                const int32_t tile = my_tile0 + P;
                const int cl = (tile - tile_wg0) * kTileN + 4 * (lane >> 4);
                if (tile < a.n_tiles)
                    *reinterpret_cast<uint32_t *>(obuf + (uint32_t)(lane & 15) * L.ostride + (uint32_t)cl) = packed;
            }
        });
    };

    for (int32_t p = p_begin, it = 0; p < p_end; ++p, ++it) {
        const int buf = it & 1;
        const int8_t *const xb = smem + (uint32_t)buf * L.xbuf;
        const int8_t *const rb = xb + (uint32_t)(lane & 15) * 32u;  // this lane's token row
        i32x4 acc[NT];
#pragma unroll
        for (int c = 0; c < NT; ++c) acc[c] = i32x4{0, 0, 0, 0};

        // Main windows: B and the index words of window w + 1 are read while
        // window w multiplies (no branches: a window past the slice multiplies
        // zero weights by the slice's first window, inside the tile). Each
        // tile's first consolidated overflow operand (or the all-zero one)
        // rides along: its header (value, index and group offsets) is read at
        // the start of window c - 1, its gathered B at the start of window c,
        // and it is multiplied after window c's matrix instructions.
        auto read_b = [&](int w) {
            const int8_t *const pb = xb + brow + (uint32_t)w * 2048u;
            const i32x4 lo = *reinterpret_cast<const i32x4 *>(pb);
            const i32x4 hi = *reinterpret_cast<const i32x4 *>(pb + 16);
            return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        };
        auto read_ix = [&](int (&ixw)[NT], int w) {
#pragma unroll
            for (int c = 0; c < NT; ++c)
                ixw[c] = *reinterpret_cast<const int *>(idxp + (uint32_t)c * idx_tile + (wbase + (uint32_t)w) * 64u);
        };
        auto ovf_first = [&](int c) { return ob[c] < oe[c] ? ob[c] : L.dummy; };
        // group offsets of the slots 8 q .. 8 q + 7 of lane group q
        auto read_go = [&](uint4 (&g)[2], uint32_t o) {
            const int8_t *const op = smem + o + kOpBytes + (lane >> 4) * 32;
            g[0] = *reinterpret_cast<const uint4 *>(op);
            g[1] = *reinterpret_cast<const uint4 *>(op + 16);
        };
        auto gather = [&](const uint4 (&g)[2]) {
            const uint32_t go[8] = {g[0].x, g[0].y, g[0].z, g[0].w, g[1].x, g[1].y, g[1].z, g[1].w};
            i32x8 bo;
#pragma unroll
            for (int j = 0; j < 8; ++j) bo[j] = *reinterpret_cast<const int *>(rb + go[j]);
            return bo;
        };
        // tile c's first overflow operand: group offsets read at the start of
        // window c - 1; gathered B, values and index words at the start of
        // window c; the product after window c's matrix instructions
        uint4 gof[2][2];
        i32x8 bv[2];
        int ixv[2][NT];
        read_go(gof[0], ovf_first(0));
        bv[0] = read_b(0);
        read_ix(ixv[0], 0);
        rs_for<NW>([&](auto wc) {
            constexpr int W = decltype(wc)::value;
            if constexpr (W + 1 < NT) read_go(gof[(W + 1) & 1], ovf_first(W + 1));
            if constexpr (W + 1 < NW) {
                bv[(W + 1) & 1] = read_b(W + 1 < nmw ? W + 1 : 0);
                read_ix(ixv[(W + 1) & 1], W + 1 < nmw ? W + 1 : 0);
            }
            i32x8 bo;
            i32x4 ao;
            int io;
            if constexpr (W < NT) {
                bo = gather(gof[W & 1]);
                const int8_t *const op = smem + ovf_first(W);
                ao = *reinterpret_cast<const i32x4 *>(op + lane * 16);
                io = *reinterpret_cast<const int *>(op + 1024 + iword * 4);
            }
#pragma unroll
            for (int c = 0; c < NT; ++c)
                acc[c] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(av[c][W], bv[W & 1], acc[c], ixv[W & 1][c], 0, 0);
            if constexpr (W < NT) acc[W] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(ao, bo, acc[W], io, 0, 0);
        });
        static_assert(NT <= NW, "every tile's first overflow operand rides along a main window");
        // further overflow operands of a tile (several only at low sparsity)
#pragma unroll
        for (int c = 0; c < NT; ++c) {
            for (uint32_t o = ob[c] + (uint32_t)kResOpBytes; o < oe[c]; o += (uint32_t)kResOpBytes) {
                uint4 g[2];
                read_go(g, o);
                const int8_t *const op = smem + o;
                const i32x4 ao = *reinterpret_cast<const i32x4 *>(op + lane * 16);
                const int io = *reinterpret_cast<const int *>(op + 1024 + iword * 4);
                acc[c] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(ao, gather(g), acc[c], io, 0, 0);
            }
        }

        int8_t *const obuf = smem + L.out + (uint32_t)buf * L.obuf;
        if (a.ks == 1) {
            if constexpr (KIND == SL_EPI_I8_GELU) {
                gelu_epilogue(acc, obuf);
            } else {
#pragma unroll
                for (int c = 0; c < NT; ++c) epilogue(acc[c], c, obuf);
            }
        } else {
            // split reduction: partials to LDS (in this pass's token tile once
            // every wave has read it, unless the tile is too small), then wave
            // kp of each channel part sums its tiles c with c % ks == kp
            int8_t *const red = smem + (L.red == 0xffffffffu ? (uint32_t)buf * L.xbuf : L.red);
            int8_t *const mine = red + (uint32_t)wave * (NT * 1024u);
            wait_lgkm0();
            __builtin_amdgcn_s_barrier();  // every wave has read the token tile
#pragma unroll
            for (int c = 0; c < NT; ++c) *reinterpret_cast<i32x4 *>(mine + c * 1024 + lane * 16) = acc[c];
            wait_lgkm0();
            __builtin_amdgcn_s_barrier();  // every partial is in LDS
            for (int c = kp; c < NT; c += a.ks) {
                i32x4 sum = i32x4{0, 0, 0, 0};
                for (int k2 = 0; k2 < a.ks; ++k2)
                    sum += *reinterpret_cast<const i32x4 *>(red + (uint32_t)(cp * a.ks + k2) * (NT * 1024u) +
                                                            (uint32_t)c * 1024u + (uint32_t)lane * 16u);
                if constexpr (KIND == SL_EPI_I8_GELU) {
                    // (one group at a time here: few groups per wave)
                    const int32_t tile = my_tile0 + c;
                    if (tile < a.n_tiles) {
#pragma clang fp contract(off)
                        const int cl = (tile - tile_wg0) * kTileN + 4 * (lane >> 4);
                        const float4 sb01 = *reinterpret_cast<const float4 *>(vec + 2 * cl);
                        const float4 sb23 = *reinterpret_cast<const float4 *>(vec + 2 * cl + 4);
                        const float s[4] = {sb01.x, sb01.z, sb23.x, sb23.z};
                        const float b[4] = {sb01.y, sb01.w, sb23.y, sb23.w};
                        const int8_t *const tabp = smem + L.tab;
                        uint32_t packed = 0;
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            float yy = (float)sum[r] * s[r];
                            yy = yy + b[r];
                            const float cf = __builtin_amdgcn_fmed3f(__builtin_fmaf(yy, hinv, goff), kGeluBase, cmax);
                            const uint2 ce = *reinterpret_cast<const uint2 *>(tabp + __umul24(__float_as_uint(cf), 8u));
                            const uint32_t q = yy >= __uint_as_float(ce.x) ? ce.y >> 8 : ce.y;
                            packed |= (q & 0xffu) << (8 * r);
                        }
                        *reinterpret_cast<uint32_t *>(obuf + (uint32_t)(lane & 15) * L.ostride + (uint32_t)cl) = packed;
                    }
                } else {
                    epilogue(sum, c, obuf);
                }
            }
        }
        // end of pass p: the staging buffer is complete for the memory wave,
        // the next token tile has landed, this one may be overwritten
        wait_lgkm0();
        __builtin_amdgcn_s_barrier();
    }
}

// ---------------------------------------------------------------------------
// host side

template <int KIND>
static sl_status launch_res_kind(const ResArgs &a, const GeluArg *ep, uint32_t grid, size_t lds, hipStream_t stream)
{
    const void *fn = reinterpret_cast<const void *>(&sparse_linear_resident_kernel<KIND>);
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
    hipLaunchKernelGGL((sparse_linear_resident_kernel<KIND>), dim3(grid), dim3(kResThreads), lds, stream, a,
                       ep ? *ep : kNoTable);
    HIP_TRY(hipGetLastError());
    return SL_OK;
}

sl_status launch_resident(const ResArgs &a, const GeluArg *ep, int32_t run_kind, uint32_t grid, size_t lds,
                          hipStream_t stream)
{
    switch (run_kind) {
    case SL_EPI_ACC_I32: return launch_res_kind<SL_EPI_ACC_I32>(a, nullptr, grid, lds, stream);
    case SL_EPI_F32: return launch_res_kind<SL_EPI_F32>(a, nullptr, grid, lds, stream);
    case SL_EPI_F32_GELU: return launch_res_kind<SL_EPI_F32_GELU>(a, nullptr, grid, lds, stream);
    case SL_EPI_I8: return launch_res_kind<SL_EPI_I8>(a, nullptr, grid, lds, stream);
    case SL_EPI_I8_GELU: return launch_res_kind<SL_EPI_I8_GELU>(a, ep, grid, lds, stream);
    default: return launch_res_kind<kEpiI8GeluErf>(a, nullptr, grid, lds, stream);
    }
}

}  // namespace sl
