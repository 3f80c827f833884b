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
//  * A workgroup owns TM tokens x NT 16-channel tiles and has two kinds of
//    waves. Copy waves stream each 128-column window into LDS with buffer
//    loads that write LDS directly: the TM input rows (the 16-byte pieces of
//    each row permuted by an XOR of the row index, so every B operand read is
//    conflict-free), the NT weight operands and the overflow operands (one
//    fixed slot per tile). Compute waves (WM x WN, each ST 16-token subtiles
//    x CT tiles) read a window's operands into registers and issue its
//    matrix instructions. Windows pass through a ring of D LDS buffers, one
//    barrier per window; while the matrix cores work on window w, the compute
//    waves read window w+1 and the copy waves fetch window w+D-1. Overflow
//    operands are read and multiplied only for tiles that have one.
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

#include "sl_device.h"

namespace sl {


// Workgroup shape: WM x WN waves; a wave owns ST 16-token subtiles x CT
// 16-channel tiles; D windows are in flight (D LDS buffers). One window's
// buffer: the TM staged token rows (128 bytes each, whole 1 KiB copies of 8
// rows), then NT main operands, then NT overflow operand slots (68 pieces of
// 16 bytes per operand). Each operand region is padded to a whole number of
// 64-lane copy instructions per wave, so every wave issues the same fixed
// number of copies per window and waits can count them.
template <int ST, int CT, int WM, int WN, int D>
struct Shape {
    static constexpr int NW = WM * WN;        // compute waves; as many copy waves again
    static constexpr int NTH = 64 * NW;       // lanes of the compute (and of the copy) waves
    static constexpr int NTHG = 2 * NTH;      // threads per workgroup
    static constexpr int TM = 16 * ST * WM;  // tokens per workgroup
    static constexpr int NT = CT * WN;       // channel tiles per workgroup
    static constexpr int XC = TM / 8;        // 1 KiB token-row copies per window
    static constexpr int CX = (XC + NW - 1) / NW;                // copies per wave: token rows
    static constexpr int CA = (NT * kOpPieces + NTH - 1) / NTH;  // copies per wave: each operand region
    static constexpr int XB = CX * NW * 1024;
    static constexpr int AB = CA * NTH * 16;
    static constexpr int COPIES = CX + 2 * CA + 1;  // per wave per window (+1: the overflow mask)
    static constexpr int BUF = XB + 2 * AB;
    static constexpr int LDS = D * BUF;
    static_assert(TM % 8 == 0, "token rows are copied 8 at a time");
};

// Position of 16-byte piece p of staged token row r: p ^ xsw(r). The 16 rows
// one B read touches then start in 16 distinct 16-byte bank groups (and any
// 8 consecutive rows in 8), so the reads are free of bank conflicts.
__device__ __forceinline__ int xsw(int r) { return (r ^ (r >> 3)) & 7; }


// VEC: X rows are 16-byte aligned and k % 16 == 0, so token rows are copied
// to LDS with 16-byte direct loads; otherwise they are staged byte by byte.
template <int KIND, int ST, int CT, int WM, int WN, int D, bool VEC, bool YT>
__device__ __forceinline__ void sparse_linear_body(const LinearArgs &a, const GeluArg *ep)
{
    using S = Shape<ST, CT, WM, WN, D>;
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    // waves 0..NW-1 read operands and run the matrix instructions; waves
    // NW..2NW-1 only issue the copies, so a copy that waits for room in the
    // memory queue never holds up the math
    const bool copier = wave >= S::NW;
    const int pw = copier ? wave - S::NW : 0;  // copy-wave index
    const int wm = wave % WM, wn = (wave / WM) % WN;

    // Work items (token tile x channel group) of this workgroup: slot,
    // slot + G, slot + 2G, ... below n_items, processed as one stream of
    // (item, window) elements through the same LDS ring: the copies of the
    // next item start while this item's last windows are multiplied, and the
    // epilogue of an item overlaps the copies of the next.
    const int32_t G = (int32_t)gridDim.x;
    const int32_t slot = (int32_t)xcd_work_index(blockIdx.x, G);
    const int n_my = (int)((a.n_items - slot + G - 1) / G);  // >= 1: the grid is at most n_items
    const int64_t steps = (int64_t)n_my * a.n_win;
    const ItemIter first = ItemIter::start(slot, G, a.n_cgroups, a.n_win);
    auto phys = [&](const ItemIter &it, int w) {
        const int p = w + it.rot;
        return p >= a.n_win ? p - a.n_win : p;
    };
    // overflow entry (mask, first index) of physical window pwin for an
    // item's tiles, from the table built at packing; the address is uniform,
    // so it is a scalar load
    typedef const __attribute__((address_space(4))) uint64_t *const_u64_ptr;
    const const_u64_ptr omt = (const_u64_ptr)(a.om);
    auto om_at = [&](const ItemIter &it, int pwin) {
        const uint64_t v = omt[(size_t)pwin * a.n_cgroups + it.cg];
        return make_uint2((uint32_t)v, (uint32_t)(v >> 32));
    };
    // overflow mask of each ring buffer's element, copied there from the
    // table by each copy wave (omask[b * NW + copy wave]) with the element's
    // operands
    uint32_t *omask = reinterpret_cast<uint32_t *>(smem + S::LDS + (KIND == SL_EPI_I8_GELU ? kGeluLds : 0) +
                                                   S::NW * kVecLds);

    GeluCell *tab = reinterpret_cast<GeluCell *>(smem + S::LDS);
    float hinv = 0.0f, eoff = 0.0f, cmax = 0.0f;
    if constexpr (KIND == SL_EPI_I8_GELU) {
        for (int u = copier ? ep->nc : tid; u < ep->nc; u += S::NTH) tab[u] = ep->cell[u];
        hinv = ep->hinv;
        eoff = ep->off;
        cmax = kGeluBase + (float)(ep->nc - 1);
    }

    // Software pipeline over the element stream, one barrier per element. In
    // step e
    //  * the copy waves wait until element e+1 has landed, pass the barrier,
    //    and start the copies of element e+D into the buffer of element e;
    //  * the compute waves pass the barrier, read element e+1's operands into
    //    one register set while the matrix instructions of element e run from
    //    the other, wait until those reads are done, and after an item's last
    //    window run its epilogue.
    // The barrier after the copy waves' wait makes element e+1 visible, and
    // means every compute wave has finished reading element e's buffer (read
    // into registers in the previous step), so D-1 elements are in flight.
    static_assert(D >= 3, "the pipeline reads one element ahead of the one it multiplies");
    static_assert((D - 1) * S::COPIES < 64, "outstanding copies must fit the 6-bit vector-memory counter");

    if (copier) {
        // Copies go through buffer loads (a lane's offset plus a scalar window
        // advance). A lane without data gets an offset past the buffer and
        // copies zeros: rows past m, operand pieces past the item's last tile,
        // absent overflow operands.
        const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
            (void *)a.x, 0, (int)min<int64_t>(a.m * a.k, kMaxBufferBytes), kRsrcWord3);
        const __amdgpu_buffer_rsrc_t mr =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.main, 0, (int)a.main_bytes, kRsrcWord3);
        const __amdgpu_buffer_rsrc_t orc =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.ovf, 0, (int)a.ovf_bytes, kRsrcWord3);
        const __amdgpu_buffer_rsrc_t omr =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.om, 0, a.n_win * a.n_cgroups * 8, kRsrcWord3);
        const uint32_t wstride = (uint32_t)a.n_tiles * kOpBytes;  // main image bytes per window
        // this lane's operand piece per operand copy
        int32_t atile[S::CA], apiece16[S::CA];
#pragma unroll
        for (int i = 0; i < S::CA; ++i) {
            const int piece = (i * S::NW + pw) * 64 + lane;
            atile[i] = piece / kOpPieces;
            apiece16[i] = (piece - atile[i] * kOpPieces) * 16;
        }

        // Element cursor: item ic (the k-th of this workgroup), window wc.
        // Past the last element it stays on the last item and repeats its
        // last window: a harmless copy that keeps the count fixed.
        ItemIter ic = first;
        int kc = 0, wc = 0;
        auto cur_w = [&]() { return phys(ic, kc < n_my ? wc : a.n_win - 1); };
        // this lane's offsets for the cursor's item: token-row copies (row
        // start + permuted piece of window 0, and the last offset inside the
        // row: a ragged last window never reads past its row, so never past
        // the buffer) and main operand copies
        uint32_t xoff[S::CX], xlim[S::CX], aoff[S::CA];
        auto item_offsets = [&]() {
            const int64_t m0 = (int64_t)ic.mt * S::TM;
            const int32_t tile0 = ic.cg * S::NT;
            const int32_t ntl = min(S::NT, a.n_tiles - tile0);
#pragma unroll
            for (int i = 0; i < S::CX; ++i) {
                const int r = ((i * S::NW + pw) * 64 + lane) / 8;
                const bool in = r < S::TM && m0 + r < a.m;
                const uint32_t row = (uint32_t)((m0 + r) * a.k);
                xoff[i] = in ? row + (uint32_t)(((lane & 7) ^ xsw(r)) * 16) : kOob;
                xlim[i] = in ? row + (uint32_t)(a.k - 16) : kOob;
            }
#pragma unroll
            for (int i = 0; i < S::CA; ++i)
                aoff[i] = atile[i] < ntl ? (uint32_t)((tile0 + atile[i]) * kOpBytes + apiece16[i]) : kOob;
        };
        auto advance = [&]() {
            if (++wc == a.n_win) {
                wc = 0;
                if (++kc < n_my) {
                    ic.next();
                    item_offsets();
                }
            }
        };
        item_offsets();

        // Copy k (0 <= k < COPIES) of the cursor's element (physical window w)
        // into ring buffer bi (global -> LDS, asynchronous): token rows, main
        // operands, the overflow mask (one lane, 4 bytes), then overflow
        // operands into the slot of their tile. o: the element's overflow
        // entry (only the overflow operand copies use it).
        constexpr int KM = S::CX + S::CA;  // the mask copy
        auto copy = [&](int k, int w, int bi, uint2 o) {
            int8_t *b = smem + bi * S::BUF;
            if (k < S::CX) {
                if constexpr (VEC)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void *)(b + (k * S::NW + pw) * 1024), 16,
                                                             min(xoff[k] + (uint32_t)(w * kWin), xlim[k]), 0, 0, 0);
            } else if (k < KM) {
                const int i = k - S::CX;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(mr, (lds_void *)(b + S::XB + (i * S::NW + pw) * 1024), 16,
                                                         aoff[i], (uint32_t)w * wstride, 0, 0);
            } else if (k == KM) {
                if (lane == 0)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(omr, (lds_void *)(omask + bi * S::NW + pw), 4,
                                                             (uint32_t)(w * a.n_cgroups + ic.cg) * 8u, 0, 0, 0);
            } else {
                const int i = k - KM - 1;
                const uint32_t mask = o.x, olo = o.y;
                const uint32_t t = (uint32_t)atile[i];
                const bool has = t < 32u && ((mask >> t) & 1u);
                const uint32_t rank = __builtin_popcount(mask & ((1u << (t & 31u)) - 1u));
                const uint32_t off = has ? (olo + rank) * (uint32_t)kOpBytes + (uint32_t)apiece16[i] : kOob;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    orc, (lds_void *)(b + S::XB + S::AB + (i * S::NW + pw) * 1024), 16, off, 0, 0, 0);
            }
        };
        // without VEC the copy waves stage the token rows by ordinary stores
        auto stage_rows = [&](int w, int8_t *b) {
            if constexpr (!VEC) {
                const int64_t m0 = (int64_t)ic.mt * S::TM;
                for (int u = tid - S::NTH; u < S::TM * kWin; u += S::NTH) {
                    const int r = u / kWin, c = u % kWin;
                    const int64_t tok = m0 + r;
                    const int32_t col = w * kWin + c;
                    b[r * kWin + (((c >> 4) ^ xsw(r)) << 4) + (c & 15)] =
                        (tok < a.m && col < a.k) ? a.x[tok * a.k + col] : (int8_t)0;
                }
            }
        };

        // Prologue: the overflow entries of elements 0..D-1 start loading, the
        // token rows, main operands and overflow masks of those elements are
        // copied, a bare barrier (A) publishes the epilogue table the compute
        // waves filled, then the overflow operands follow; once element 0 has
        // landed a second barrier (B) publishes it.
        uint2 o[D];
        {
            const ItemIter ic0 = ic;
            const int kc0 = kc, wc0 = wc;
#pragma unroll
            for (int d = 0; d < D; ++d) {
                o[d] = om_at(ic, cur_w());
                if (++wc == a.n_win) {
                    wc = 0;
                    if (++kc < n_my) ic.next();
                }
            }
            ic = ic0;
            kc = kc0;
            wc = wc0;
        }
        int wp[D];
#pragma unroll
        for (int d = 0; d < D; ++d) {
            wp[d] = cur_w();
#pragma unroll
            for (int k = 0; k <= KM; ++k) copy(k, wp[d], d, make_uint2(0u, 0u));
            stage_rows(wp[d], smem + d * S::BUF);
            advance();
        }
        __builtin_amdgcn_s_barrier();  // (A)
        asm volatile("" ::: "memory");
#pragma unroll
        for (int d = 0; d < D; ++d) {
#pragma unroll
            for (int k = KM + 1; k < S::COPIES; ++k) copy(k, wp[d], d, o[d]);
        }
        uint2 onx = om_at(ic, cur_w());  // entry of element D
        if constexpr (VEC)
            wait_vmcnt_le<(D - 1) * S::CA>();  // element 0 landed
        else
            __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_s_barrier();  // (B)
        asm volatile("" ::: "memory");

        // step e: copies of element e+D into the buffer of element e; the
        // overflow entry of the next element loads across the next barrier
        auto cstep = [&](int64_t e, int u) {
            if (e + 1 < steps) {
                if constexpr (VEC)
                    wait_window_landed<D, S::CA, S::COPIES>((int)(e < D ? e : D));
                else
                    __builtin_amdgcn_s_waitcnt(0);
            }
            // a bare barrier: __syncthreads() would also wait for the later
            // elements' copies still in flight
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            const int b = u;
            const int w = cur_w();
#pragma unroll
            for (int k = 0; k < S::COPIES; ++k) copy(k, w, b, onx);
            stage_rows(w, smem + b * S::BUF);
            advance();
            onx = om_at(ic, cur_w());
        };
        constexpr int U = D;  // unroll: the buffer index repeats
        int64_t e = 0;
        for (; e + U <= steps; e += U) {
#pragma unroll
            for (int u = 0; u < U; ++u) cstep(e + u, u);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (e + u < steps) cstep(e + u, u);
        __builtin_amdgcn_s_waitcnt(0);  // no copy may land after the workgroup ends
        return;
    }
    __builtin_amdgcn_s_waitcnt(0);  // the epilogue table's LDS stores are done
    __builtin_amdgcn_s_barrier();   // (A)
    asm volatile("" ::: "memory");

    // ---- compute waves

    // this lane's B rows (token (lane & 15) of each subtile) and 32-column
    // slice of the window: pieces 2h and 2h+1, h = lane / 16
    int brow[ST][2];
#pragma unroll
    for (int s = 0; s < ST; ++s) {
        const int r = wm * ST * 16 + s * 16 + (lane & 15);
        const int p0 = 2 * (lane >> 4);
        brow[s][0] = r * kWin + ((p0 ^ xsw(r)) << 4);
        brow[s][1] = r * kWin + (((p0 + 1) ^ xsw(r)) << 4);
    }
    // this lane's index word: block-row (lane%16)/4, lane group lane/16
    const int iword = ((lane & 15) >> 2) * 4 + (lane >> 4);

    // Operands of one element in registers: B (token rows), main and overflow
    // A operands with their index words. Two sets alternate (steps e, e+1).
    struct Ops {
        i32x8 bv[ST];
        i32x4 av[CT], ao[CT];
        int ix[CT], io[CT];
    };
    Ops ops[2];
    // main operands (B rows, main A and index words) of one element
    auto read_main = [&](Ops &r, const int8_t *b) {
#pragma unroll
        for (int s = 0; s < ST; ++s) {
            const i32x4 lo = *reinterpret_cast<const i32x4 *>(b + brow[s][0]);
            const i32x4 hi = *reinterpret_cast<const i32x4 *>(b + brow[s][1]);
            r.bv[s] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
#pragma unroll
        for (int c = 0; c < CT; ++c) {
            const int8_t *op = b + S::XB + (wn * CT + c) * kOpBytes;
            r.av[c] = *reinterpret_cast<const i32x4 *>(op + lane * 16);
            r.ix[c] = *reinterpret_cast<const int *>(op + 1024 + iword * 4);
        }
    };
    // overflow operand of tile c of one element (read only if the tile has one)
    auto read_ovf = [&](Ops &r, const int8_t *b, int c) {
        const int8_t *oo = b + S::XB + S::AB + (wn * CT + c) * kOpBytes;
        r.ao[c] = *reinterpret_cast<const i32x4 *>(oo + lane * 16);
        r.io[c] = *reinterpret_cast<const int *>(oo + 1024 + iword * 4);
    };
    auto read_mask = [&](int b) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)omask[b * S::NW]); };

    // This wave's weight scales and biases of an item (CT tiles x 16 channels
    // each) go into its own LDS area with one copy per vector at the item's
    // first window; the epilogue reads them after waiting for its own copies.
    float *vec = reinterpret_cast<float *>(smem + S::LDS + (KIND == SL_EPI_I8_GELU ? kGeluLds : 0) + wave * kVecLds);
    static_assert(CT * kTileN * 4 <= kVecLds / 2, "a wave's scales fit one copy");
    auto fetch_vec = [&](const ItemIter &it) {
        if constexpr (KIND != SL_EPI_ACC_I32) {
            const __amdgpu_buffer_rsrc_t sr =
                __builtin_amdgcn_make_buffer_rsrc((void *)a.w_scale, 0, a.n * 4, kRsrcWord3);
            const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc((void *)a.bias, 0, a.n * 4, kRsrcWord3);
            // only the first CT*4 lanes copy (16 bytes each), so a copy fills
            // CT*64 bytes of LDS
            if (lane < CT * 4) {
                const uint32_t off = (uint32_t)(((it.cg * S::NT + wn * CT) * kTileN + lane * 4) * 4);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(sr, (lds_void *)vec, 16, off, 0, 0, 0);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(br, (lds_void *)(vec + kVecLds / 8), 16, off, 0, 0, 0);
            }
        }
    };

    i32x4 acc[CT][ST];
    auto clear_acc = [&]() {
#pragma unroll
        for (int c = 0; c < CT; ++c)
#pragma unroll
            for (int s = 0; s < ST; ++s) acc[c][s] = i32x4{0, 0, 0, 0};
    };
    // accumulator layout: lane l holds rows 4*(l/16)+r (channels of one
    // block-row), column l%16 (token), r = 0..3
    auto epilogue = [&](const ItemIter &it) {
        __builtin_amdgcn_s_waitcnt(0);  // this wave's scale and bias copies
        const int64_t m0 = (int64_t)it.mt * S::TM;
#pragma unroll
        for (int c = 0; c < CT; ++c) {
            const int32_t t = it.cg * S::NT + wn * CT + c;
            if (t >= a.n_tiles) break;
            const int32_t ch0 = t * kTileN + 4 * (lane >> 4);
            if (ch0 >= a.n) continue;  // block-rows past n_out in the last tile
            float s[4] = {0, 0, 0, 0}, bb4[4] = {0, 0, 0, 0};
            if constexpr (KIND != SL_EPI_ACC_I32) {
                const int lc = c * kTileN + 4 * (lane >> 4);  // channel within the wave's tiles
                const float4 sw = *reinterpret_cast<const float4 *>(vec + lc);
                const float4 bb = *reinterpret_cast<const float4 *>(vec + kVecLds / 8 + lc);
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
                epilogue_store<KIND, YT>(a, acc[c][st], m0 + wm * ST * 16 + st * 16 + (lane & 15), ch0, s, bb4, tab, hinv,
                                     eoff, cmax);
        }
    };

    // sl: ring buffer of element e; mask_w: overflow mask of element e (its
    // operands are in register set PR)
    int sl = 0;
    int64_t e = 0;
    uint32_t mask_w;
    auto step = [&](auto pr) {
        constexpr int PR = decltype(pr)::value;
        Ops &cur = ops[PR];
        Ops &nxt = ops[PR ^ 1];
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        const int sl1 = sl + 1 == D ? 0 : sl + 1;
        const int8_t *nb = smem + sl1 * S::BUF;
        // Main part: element e+1's main operand reads and element e's main
        // matrix instructions, one after the other, so that a read waiting
        // for room in the LDS queue does not leave the matrix core idle.
        // (The last step reads a stale buffer: harmless, and branch-free.)
        // Main products of tiles past the item's last tile land in
        // accumulators that are never stored, so they need no branch either.
        read_main(nxt, nb);
#pragma unroll
        for (int c = 0; c < CT; ++c)
#pragma unroll
            for (int s = 0; s < ST; ++s)
                acc[c][s] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(cur.av[c], cur.bv[s], acc[c][s], cur.ix[c], 0, 0);
#pragma unroll
        for (int v = 0; v < CT * ST; ++v) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one matrix instruction
        }
        __builtin_amdgcn_sched_group_barrier(0x100, 2 * ST + 2 * CT, 0);  // the remaining reads
        // element e+1's overflow mask, read once the main matrix instructions
        // are queued (its latency hides behind them)
        __builtin_amdgcn_sched_barrier(0);
        const uint32_t mask_n = read_mask(sl1);
        // overflow part, per tile
#pragma unroll
        for (int c = 0; c < CT; ++c) {
            const int jw = wn * CT + c;
            if (e + 1 < steps && ((mask_n >> jw) & 1u)) read_ovf(nxt, nb, c);
            if ((mask_w >> jw) & 1u) {
#pragma unroll
                for (int s = 0; s < ST; ++s)
                    acc[c][s] =
                        __builtin_amdgcn_smfmac_i32_16x16x128_i8(cur.ao[c], cur.bv[s], acc[c][s], cur.io[c], 0, 0);
            }
        }
        // element e+1's buffer is refilled after the next barrier: its
        // reads must be done by then
        wait_lgkm0();
        mask_w = mask_n;
        sl = sl1;
        ++e;
    };
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;

    ItemIter it = first;
    clear_acc();
    fetch_vec(it);
    __builtin_amdgcn_s_barrier();  // (B): element 0 has landed
    asm volatile("" ::: "memory");
    mask_w = read_mask(0);
    read_main(ops[0], smem);
#pragma unroll
    for (int c = 0; c < CT; ++c)
        if ((mask_w >> (wn * CT + c)) & 1u) read_ovf(ops[0], smem, c);
    wait_lgkm0();  // element 0's buffer is refilled after the next barrier
    // Each item starts with its first element's operands in register set 0;
    // after an odd number of windows they are moved there from set 1.
    for (int k = 0; k < n_my; ++k) {
        int w = 0;
        for (; w + 2 <= a.n_win; w += 2) {
            step(P0{});
            step(P1{});
        }
        if (w < a.n_win) {
            step(P0{});
            ops[0] = ops[1];
        }
        epilogue(it);
        if (k + 1 < n_my) {
            clear_acc();
            it.next();
            asm volatile("" ::: "memory");  // the epilogue's reads of the scales come first
            fetch_vec(it);
        }
    }
}

template <int KIND, int ST, int CT, int WM, int WN, int D, bool VEC, bool YT>
__global__ __launch_bounds__(128 * WM * WN) void sparse_linear_kernel(LinearArgs a)
{
    sparse_linear_body<KIND, ST, CT, WM, WN, D, VEC, YT>(a, nullptr);
}

template <int ST, int CT, int WM, int WN, int D, bool VEC, bool YT>
__global__ __launch_bounds__(128 * WM * WN) void sparse_linear_gelu_kernel(LinearArgs a, GeluArg ep)
{
    sparse_linear_body<SL_EPI_I8_GELU, ST, CT, WM, WN, D, VEC, YT>(a, &ep);
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
        store_nt(reinterpret_cast<uint4 *>(q) + i, o);
    }
}

__global__ __launch_bounds__(256) void quantize_scalar_kernel(const float *x, int64_t n, float inv, int8_t *q)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        q[i] = (int8_t)requant_i8(x[i], inv);
}

// Quantisation into the 16-token x 32-feature block layout: thread j writes
// 16-byte piece j of the output (block j / 32; token (j % 32) / 2 of the
// block, features 16 * (j % 2) .. +15 of the block's 32), zeros for padding.
// VEC: cols % 4 == 0 and x 16-byte aligned, so whole pieces load as float4.
template <bool VEC>
__global__ __launch_bounds__(256) void quantize_t16x32_kernel(const float *x, int64_t rows, int32_t cols,
                                                              int32_t cblocks, int64_t n_pieces, float inv,
                                                              int8_t *q)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n_pieces; j += stride) {
        const int64_t b = j >> 5;
        const int w = (int)(j & 31);
        const int64_t t = (b / cblocks) * 16 + (w >> 1);
        const int32_t c0 = (int32_t)(b % cblocks) * 32 + (w & 1) * 16;
        uint4 o = {0u, 0u, 0u, 0u};
        if (t < rows) {
            const float *row = x + t * cols;
            if (VEC && c0 + 16 <= cols) {
                const float4 *src = reinterpret_cast<const float4 *>(row + c0);
                o.x = quant4(src[0], inv);
                o.y = quant4(src[1], inv);
                o.z = quant4(src[2], inv);
                o.w = quant4(src[3], inv);
            } else {
                uint32_t v[4] = {0u, 0u, 0u, 0u};
                for (int i = 0; i < 16 && c0 + i < cols; ++i)
                    v[i >> 2] |= ((uint32_t)requant_i8(row[c0 + i], inv) & 0xffu) << (8 * (i & 3));
                o = make_uint4(v[0], v[1], v[2], v[3]);
            }
        }
        store_nt(reinterpret_cast<uint4 *>(q) + j, o);
    }
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
        set_error("device %d is %s; this library has gfx950 kernels only", dev, prop.gcnArchName);
        return SL_ERR_UNSUPPORTED;
    }
    *device = dev;
    return SL_OK;
}

// Workgroup shapes (ST, CT, WM, WN, D): (16*ST*WM) tokens x (16*CT*WN)
// channels, D windows in flight.
struct TileCfg {
    int st, ct, wm, wn, d;
    int tm() const { return 16 * st * wm; }
    int nt() const { return ct * wn; }
};
static const TileCfg kCfgs[] = {
    {4, 3, 2, 2, 3},  // 128 x  96,  96 KiB LDS
    {4, 3, 2, 2, 4},  // 128 x  96, 128 KiB
    {2, 3, 2, 2, 3},  //  64 x  96,  72 KiB (two workgroups per CU)
    {2, 3, 2, 2, 4},  //  64 x  96,  96 KiB
    {1, 3, 2, 2, 6},  //  32 x  96, 120 KiB (few tokens: deep ring)
    {1, 1, 2, 2, 8},  //  32 x  32,  96 KiB (few tokens: deep ring)
};

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

sl_status upload_image(sl_packed_weight *w)
{
    const TileImage &ti = w->tiles;
    if ((int64_t)ti.main.size() > kMaxBufferBytes || (int64_t)ti.ovf.size() > kMaxBufferBytes) {
        set_error("packed weight image over 2 GiB (n_out x k_in too large for one image)");
        return SL_ERR_UNSUPPORTED;
    }
    // overflow tables, one per tile-group size of the staged kernel's shapes
    std::vector<int> nts;
    for (const TileCfg &c : kCfgs)
        if (std::find(nts.begin(), nts.end(), c.nt()) == nts.end()) nts.push_back(c.nt());
    if ((int)nts.size() > kMaxOmTables) {
        set_error("internal: too many tile-group sizes");
        return SL_ERR_UNSUPPORTED;
    }
    std::vector<std::vector<uint32_t>> oms(nts.size());
    const size_t pstride = (size_t)ti.n_tiles + 1;
    for (size_t i = 0; i < nts.size(); ++i) {
        const int nt = nts[i];
        const int ncg = (ti.n_tiles + nt - 1) / nt;
        std::vector<uint32_t> &om = oms[i];
        om.assign((size_t)ti.n_win * ncg * 2, 0u);
        for (int wi = 0; wi < ti.n_win; ++wi)
            for (int g = 0; g < ncg; ++g) {
                const int t0 = g * nt, ntl = std::min(nt, ti.n_tiles - t0);
                const uint32_t *pp = ti.ovf_ptr.data() + (size_t)wi * pstride + t0;
                uint32_t mask = 0;
                for (int j = 0; j < ntl; ++j) mask |= (pp[j + 1] > pp[j] ? 1u : 0u) << j;
                om[((size_t)wi * ncg + g) * 2] = mask;
                om[((size_t)wi * ncg + g) * 2 + 1] = pp[0];
            }
    }
    // weight panels, one table per tile-group size of the weight-stationary shapes
    std::vector<int> pnts;
    for (const PanelCfg &c : kPanelCfgs)
        if (std::find(pnts.begin(), pnts.end(), c.nt) == pnts.end()) pnts.push_back(c.nt);
    if ((int)pnts.size() > kMaxPanTables) {
        set_error("internal: too many weight-panel sizes");
        return SL_ERR_UNSUPPORTED;
    }
    std::vector<std::vector<uint32_t>> pans(pnts.size());
    std::vector<uint32_t> pan_max(pnts.size(), 0);
    for (size_t i = 0; i < pnts.size(); ++i) {
        const int nt = pnts[i];
        const int ncg = (ti.n_tiles + nt - 1) / nt;
        std::vector<uint32_t> &pt = pans[i];
        pt.assign((size_t)ncg * (ti.n_win + 1) * 4, 0u);
        for (int g = 0; g < ncg; ++g) {
            const int t0 = g * nt, ntl = std::min(nt, ti.n_tiles - t0);
            uint64_t base = 0;
            for (int wi = 0; wi < ti.n_win; ++wi) {
                const uint32_t *pp = ti.ovf_ptr.data() + (size_t)wi * pstride + t0;
                uint32_t mask = 0;
                for (int j = 0; j < ntl; ++j) mask |= (pp[j + 1] > pp[j] ? 1u : 0u) << j;
                uint32_t *e = &pt[((size_t)g * (ti.n_win + 1) + wi) * 4];
                e[0] = mask;
                e[1] = pp[0];
                e[2] = (uint32_t)std::min<uint64_t>(base, UINT32_MAX);
                base += (uint64_t)(2 * nt) * kOpPieces;
            }
            pt[((size_t)g * (ti.n_win + 1) + ti.n_win) * 4 + 2] = (uint32_t)std::min<uint64_t>(base, UINT32_MAX);
            pan_max[i] = (uint32_t)std::min<uint64_t>(std::max<uint64_t>(pan_max[i], base), UINT32_MAX);
        }
    }
    // The panel images: per channel group, its window table and then its
    // panel (per window: the NT main operands, zeros past the last tile, then
    // NT overflow operand slots, zeros where a tile has none), padded to a
    // common stride of whole 1024-byte copies, so that a workgroup's copies
    // need no table read first and its kernel none at all.
    // Only sizes whose panels can fit in LDS get an image.
    std::vector<std::vector<int8_t>> pimgs(pnts.size());
    std::vector<uint32_t> pstrides(pnts.size(), 0);
    for (size_t i = 0; i < pnts.size(); ++i) {
        const int nt = pnts[i];
        const int ncg = (ti.n_tiles + nt - 1) / nt;
        const uint64_t tab = (uint64_t)(ti.n_win + 1) * 16;
        const uint64_t stride = (tab + (uint64_t)pan_max[i] * 16 + 1023) / 1024 * 1024;
        if (stride > kLdsMax || (uint64_t)ncg * stride > (uint64_t)kMaxBufferBytes) continue;
        pstrides[i] = (uint32_t)stride;
        std::vector<int8_t> &im = pimgs[i];
        im.assign((size_t)ncg * stride, 0);
        const std::vector<uint32_t> &pt = pans[i];
        for (int g = 0; g < ncg; ++g) {
            int8_t *const gb = im.data() + (size_t)g * stride;
            const uint32_t *const ge = pt.data() + (size_t)g * (ti.n_win + 1) * 4;
            memcpy(gb, ge, (size_t)tab);
            const int t0 = g * nt, ntl = std::min(nt, ti.n_tiles - t0);
            for (int wi = 0; wi < ti.n_win; ++wi) {
                int8_t *const wb = gb + tab + (size_t)ge[wi * 4 + 2] * 16;
                memcpy(wb, ti.main.data() + ((size_t)wi * ti.n_tiles + t0) * kOpBytes, (size_t)ntl * kOpBytes);
                // (the window's overflow operands are stored in tile order
                // from entry word 1 on)
                uint32_t rank = 0;
                for (int j = 0; j < ntl; ++j)
                    if ((ge[wi * 4] >> j) & 1u) {
                        memcpy(wb + (size_t)(nt + j) * kOpBytes,
                               ti.ovf.data() + (size_t)(ge[wi * 4 + 1] + rank) * kOpBytes, kOpBytes);
                        ++rank;
                    }
            }
        }
    }
    // the dense overflow image of the split-reduction and direct kernels: a
    // tile's overflow operand of a window at the offset of its main operand,
    // zeros where it has none (the same size as the main image, which is
    // known to fit one buffer)
    std::vector<int8_t> odense(ti.main.size(), 0);
    {
        const size_t pstride = (size_t)ti.n_tiles + 1;
        for (int wi = 0; wi < ti.n_win; ++wi)
            for (int t = 0; t < ti.n_tiles; ++t) {
                const uint32_t *pp = ti.ovf_ptr.data() + (size_t)wi * pstride + t;
                if (pp[1] > pp[0])
                    memcpy(odense.data() + ((size_t)wi * ti.n_tiles + t) * kOpBytes,
                           ti.ovf.data() + (size_t)pp[0] * kOpBytes, kOpBytes);
            }
    }
    const size_t b_main = std::max<size_t>(ti.main.size(), 16);
    const size_t b_ovf = std::max<size_t>(ti.ovf.size(), 16);
    const size_t b_vec = (size_t)w->n_out * sizeof(float);
    const size_t o_main = 0;
    const size_t o_ovf = align256(o_main + b_main);
    const size_t o_sw = align256(o_ovf + b_ovf);
    const size_t o_b = align256(o_sw + b_vec);
    size_t o_end = align256(o_b + b_vec);
    std::vector<size_t> o_om(nts.size());
    for (size_t i = 0; i < nts.size(); ++i) {
        o_om[i] = o_end;
        o_end = align256(o_end + oms[i].size() * sizeof(uint32_t));
    }
    std::vector<size_t> o_pan(pnts.size());
    for (size_t i = 0; i < pnts.size(); ++i) {
        o_pan[i] = o_end;
        o_end = align256(o_end + pimgs[i].size());
    }
    const size_t o_ovfd = o_end;
    o_end = align256(o_end + b_main);
    const size_t total = o_end;
    void *base = nullptr;
    hipError_t e = hipMalloc(&base, total);
    if (e != hipSuccess) {
        set_error("hipMalloc of the packed weight: %s", hipGetErrorString(e));
        return e == hipErrorOutOfMemory ? SL_ERR_OOM : SL_ERR_HIP;
    }
    char *p = static_cast<char *>(base);
    w->dev.base = base;
    w->dev.bytes = (int64_t)total;
    w->on_device = true;  // from here on sparse_linear_free releases the memory
    if (!ti.main.empty()) HIP_TRY(hipMemcpy(p + o_main, ti.main.data(), ti.main.size(), hipMemcpyHostToDevice));
    if (!ti.ovf.empty()) HIP_TRY(hipMemcpy(p + o_ovf, ti.ovf.data(), ti.ovf.size(), hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p + o_sw, w->w_scale.data(), b_vec, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p + o_b, w->bias.data(), b_vec, hipMemcpyHostToDevice));
    for (size_t i = 0; i < nts.size(); ++i) {
        HIP_TRY(hipMemcpy(p + o_om[i], oms[i].data(), oms[i].size() * sizeof(uint32_t), hipMemcpyHostToDevice));
        w->dev.om_nt[i] = nts[i];
        w->dev.om[i] = reinterpret_cast<const uint32_t *>(p + o_om[i]);
    }
    w->dev.n_om = (int32_t)nts.size();
    for (size_t i = 0; i < pnts.size(); ++i) {
        if (!pimgs[i].empty())
            HIP_TRY(hipMemcpy(p + o_pan[i], pimgs[i].data(), pimgs[i].size(), hipMemcpyHostToDevice));
        w->dev.pan_nt[i] = pnts[i];
        w->dev.pan_pieces[i] = (int32_t)std::min<uint32_t>(pan_max[i], INT32_MAX);
        w->dev.pan_stride[i] = pstrides[i];
        w->dev.pan[i] = pimgs[i].empty() ? nullptr : reinterpret_cast<const int8_t *>(p + o_pan[i]);
    }
    w->dev.n_pan = (int32_t)pnts.size();
    if (!odense.empty()) HIP_TRY(hipMemcpy(p + o_ovfd, odense.data(), odense.size(), hipMemcpyHostToDevice));
    w->dev.ovfd = reinterpret_cast<const int8_t *>(p + o_ovfd);
    w->dev.ovfd_bytes = (uint32_t)odense.size();
    w->dev.main = reinterpret_cast<const int8_t *>(p + o_main);
    w->dev.ovf = reinterpret_cast<const int8_t *>(p + o_ovf);
    w->dev.ovf_ptr = nullptr;
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

sl_status persistent_grid(const void *fn, int threads, size_t lds, int *cache, int *out)
{
    int dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) {
        set_error("device index beyond the supported range");
        return SL_ERR_UNSUPPORTED;
    }
    // a benign race: two threads may both fill the entry, with equal values
    if (!cache[dev]) {
        HIP_TRY(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax));
        int per_cu = 0, n_cu = 0;
        HIP_TRY(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev));
        HIP_TRY(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, lds));
        cache[dev] = std::max(1, per_cu) * std::max(1, n_cu);
    }
    *out = cache[dev];
    return SL_OK;
}

template <int KIND, int ST, int CT, int WM, int WN, int D, bool VEC, bool YT>
static sl_status launch_cfg(const LinearArgs &a, const GeluArg *ep, hipStream_t stream)
{
    using S = Shape<ST, CT, WM, WN, D>;
    const void *fn;
    if constexpr (KIND == SL_EPI_I8_GELU)
        fn = reinterpret_cast<const void *>(&sparse_linear_gelu_kernel<ST, CT, WM, WN, D, VEC, YT>);
    else
        fn = reinterpret_cast<const void *>(&sparse_linear_kernel<KIND, ST, CT, WM, WN, D, VEC, YT>);
    const size_t lds = (size_t)S::LDS + S::NW * kVecLds + kMaskLds + (KIND == SL_EPI_I8_GELU ? kGeluLds : 0);
    static_assert(S::LDS + S::NW * kVecLds + kMaskLds + kGeluLds <= kLdsMax, "workgroup shape exceeds LDS");
    static_assert(D * S::NW * 4 <= kMaskLds, "one overflow mask per ring buffer and copy wave");
    // persistent grid: as many workgroups as fit on the device at once, each
    // taking every G-th work item
    static int resident[kMaxDevices] = {};  // per kernel instance and device
    int grid = 0;
    const sl_status st = persistent_grid(fn, S::NTHG, lds, resident, &grid);
    if (st != SL_OK) return st;
    const int64_t nwg = std::min<int64_t>(a.n_items, grid);
    if constexpr (KIND == SL_EPI_I8_GELU)
        hipLaunchKernelGGL((sparse_linear_gelu_kernel<ST, CT, WM, WN, D, VEC, YT>), dim3((uint32_t)nwg), dim3(S::NTHG),
                           lds, stream, a, *ep);
    else
        hipLaunchKernelGGL((sparse_linear_kernel<KIND, ST, CT, WM, WN, D, VEC, YT>), dim3((uint32_t)nwg), dim3(S::NTHG),
                           lds, stream, a);
    HIP_TRY(hipGetLastError());
    return SL_OK;
}

template <int KIND, bool VEC, bool YT>
static sl_status launch_kind(const LinearArgs &a, const GeluArg *ep, TileCfg c, hipStream_t stream)
{
#define SL_CFG(A_, B_, C_, D_, E_)                                         \
    if (c.st == A_ && c.ct == B_ && c.wm == C_ && c.wn == D_ && c.d == E_) \
        return launch_cfg<KIND, A_, B_, C_, D_, E_, VEC, YT>(a, ep, stream);
    SL_CFG(4, 3, 2, 2, 3)
    SL_CFG(4, 3, 2, 2, 4)
    SL_CFG(2, 3, 2, 2, 3)
    SL_CFG(2, 3, 2, 2, 4)
    SL_CFG(1, 3, 2, 2, 6)
#undef SL_CFG
    return launch_cfg<KIND, 1, 1, 2, 2, 8, VEC, YT>(a, ep, stream);
}

// The staged kernel writes the block layout only for rows the direct kernel
// cannot load (k_in % 16 != 0 or a misaligned x): int8 kinds without VEC.
template <int KIND>
static sl_status launch_vec(const LinearArgs &a, const GeluArg *ep, TileCfg c, hipStream_t stream, bool vec, bool yt)
{
    if constexpr (EpiOut<KIND>::kBytes == 1) {
        if (yt) {
            if (vec) {
                set_error("internal: aligned rows with a block-layout output go through the direct kernel");
                return SL_ERR_UNSUPPORTED;
            }
            return launch_kind<KIND, false, true>(a, ep, c, stream);
        }
    }
    return vec ? launch_kind<KIND, true, false>(a, ep, c, stream) : launch_kind<KIND, false, false>(a, ep, c, stream);
}

// Pick the workgroup shape: among shapes that give every CU a workgroup,
// the one with the least L2 traffic (token rows re-read once per channel
// group, the weight image once per token group); SL_TILE="st,ct,wm,wn,d"
// overrides (tuning; unknown shapes are ignored).
static TileCfg choose_cfg(int64_t m, const sl_packed_weight *w)
{
    const int *e = env_cfg().tile;
    if (e[0])
        for (const TileCfg &k : kCfgs)
            if (k.st == e[0] && k.ct == e[1] && k.wm == e[2] && k.wn == e[3] && k.d == e[4]) return k;
    const int32_t n_tiles = w->tiles.n_tiles;
    const double xbytes = (double)m * w->k_in;
    const double wbytes = (double)w->tiles.main.size() + (double)w->tiles.ovf.size();
    const TileCfg *best = nullptr, *most = nullptr;
    double best_cost = 0;
    int64_t most_wg = 0;
    for (const TileCfg &c : kCfgs) {
        if (c.d != 4 || c.wm * c.wn != 4) continue;
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

// Direct-kernel shape, by the same rule; SL_DTILE="st,nt,wm,d" overrides.
static DirectCfg choose_direct_cfg(int64_t m, const sl_packed_weight *w)
{
    const int *e = env_cfg().dtile;
    if (e[0])
        for (const DirectCfg &k : kDirectCfgs)
            if (k.st == e[0] && k.nt == e[1] && k.wm == e[2] && k.d == e[3]) return k;
    const int32_t n_tiles = w->tiles.n_tiles;
    const double xbytes = (double)m * w->k_in;
    const double wbytes = (double)w->tiles.main.size() + (double)w->tiles.ovf.size();
    const DirectCfg *best = nullptr, *most = nullptr;
    double best_cost = 0;
    int64_t most_items = 0;
    for (const DirectCfg &c : kDirectCfgs) {
        const int64_t mt = (m + c.tm() - 1) / c.tm();
        const int64_t cgs = (n_tiles + c.nt - 1) / c.nt;
        const int64_t items = mt * cgs;
        if (items > most_items) {
            most_items = items;
            most = &c;
        }
        if (items < 240) continue;
        const double cost = xbytes * cgs + wbytes * mt;
        if (!best || cost < best_cost) {
            best = &c;
            best_cost = cost;
        }
    }
    return best ? *best : *most;
}

// The default path takes the weight-stationary kernel only for reductions
// of at most this many 128-feature windows (K <= 1024).
constexpr int32_t kPanelMaxWin = 8;

// Whether the work items of the kernel that runs where the weight-stationary
// one does not (direct, else staged) make one round of the CUs that keeps at
// least 80 % of them busy. Over short reductions that kernel wins only
// there: a second round costs a whole item's time again, where the
// weight-stationary kernel reuses its panel.
static bool one_full_round(bool direct, int64_t m, const sl_packed_weight *w)
{
    int dev = 0, n_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n_cu < 1)
        return true;
    int64_t tm, nt;
    if (direct) {
        const DirectCfg c = choose_direct_cfg(m, w);
        tm = c.tm();
        nt = c.nt;
    } else {
        const TileCfg c = choose_cfg(m, w);
        tm = c.tm();
        nt = c.nt();
    }
    const int64_t items = (m + tm - 1) / tm * ((w->tiles.n_tiles + nt - 1) / nt);
    return items <= n_cu && items * 5 >= (int64_t)n_cu * 4;
}

// Weight-stationary shape for a launch of a.m tokens: the compiled shapes
// whose largest panel fits in LDS are scored by the bytes their workgroups
// read (token rows once per channel group, the panel once per workgroup)
// spread over the CUs they keep busy, with a small preference for more
// resident waves a SIMD; SL_PTILE="nt,st,nwv,r" overrides the shape and
// SL_PSLICES=n the number of token slices (tests: many token groups a wave
// at small sizes). Fills a's channel-group and slice fields;
// SL_ERR_UNSUPPORTED when no panel fits.
static sl_status choose_panel_cfg(LinearArgs &a, const sl_packed_weight *w, int32_t run_kind, bool yt, PanelCfg *out,
                                  size_t *lds_out)
{
    int n_cu = 0, dev = 0;
    HIP_TRY(hipGetDevice(&dev));
    HIP_TRY(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev));
    const int *e = env_cfg().ptile;
    const PanelCfg forced{e[0], e[1], e[2], e[3]};
    const bool have_forced = e[0] != 0;
    const int64_t mpad = (a.m + 15) / 16 * 16;
    double best_cost = 0;
    bool found = false;
    for (int ci = 0; ci < kNumPanelCfgs; ++ci) {
        const PanelCfg c = kPanelCfgs[ci];
        if (have_forced && (c.nt != forced.nt || c.st != forced.st || c.nwv != forced.nwv || c.r != forced.r))
            continue;
        int pi = -1;
        for (int i = 0; i < w->dev.n_pan; ++i)
            if (w->dev.pan_nt[i] == c.nt) pi = i;
        if (pi < 0 || !w->dev.pan_stride[pi]) continue;
        const int32_t pieces = w->dev.pan_pieces[pi];
        const size_t lds = panel_lds_bytes(c, run_kind, yt, w->dev.pan_stride[pi]);
        if (lds > kLdsMax) continue;
        // resident workgroups per device, cached per (device, shape, LDS size)
        static thread_local struct {
            int dev, ci;
            size_t lds;
            int res;
        } cache[16];
        static thread_local int cache_n = 0;
        int res = -1;
        for (int i = 0; i < cache_n; ++i)
            if (cache[i].dev == dev && cache[i].ci == ci && cache[i].lds == lds) res = cache[i].res;
        if (res < 0) {
            const sl_status st = panel_resident(c, lds, &res);
            if (st != SL_OK) return st;
            cache[cache_n % 16] = {dev, ci, lds, res};
            cache_n = cache_n < 16 ? cache_n + 1 : 16;
        }
        if (res < 1) continue;
        const int64_t n_cg = (w->tiles.n_tiles + c.nt - 1) / c.nt;
        const int64_t groups = (mpad + c.tg() - 1) / c.tg();
        // slices: enough workgroups to fill the resident slots once, or one
        // workgroup a CU (fewer panel fills, more token groups a wave),
        // whichever scores better
        for (int64_t want : {res / n_cg, (int64_t)n_cu / n_cg}) {
            want = std::max<int64_t>(1, env_cfg().pslices > 0 ? env_cfg().pslices : want);
            const int64_t sg = std::max<int64_t>(1, (groups + want - 1) / want);
            const int64_t n_sl = (groups + sg - 1) / sg;
            const int64_t nwg = n_cg * n_sl;
            if (nwg > 0x7fffffff) continue;
            // busy CUs and the bytes each reads
            const double cus = (double)std::min<int64_t>(n_cu, nwg);
            const double bytes = (double)a.m * w->k_in * n_cg + (double)nwg * pieces * 16.0;
            // waves per workgroup without a token group idle; among shapes
            // that read the same bytes, more resident waves a SIMD hide more
            // latency
            const double wave_use = std::min(1.0, (double)sg / c.nwv);
            const double simd_waves = std::min(4.0, (double)std::min<int64_t>(res, nwg) / n_cu * c.nwv / 4.0);
            const double cost = bytes / cus / wave_use / (1.0 + 0.1 * simd_waves);
            if (!found || cost < best_cost) {
                found = true;
                best_cost = cost;
                *out = c;
                *lds_out = lds;
                a.n_cgroups = (int32_t)n_cg;
                a.n_slices = (int32_t)n_sl;
                a.slice_groups = (int32_t)sg;
                a.pan = w->dev.pan[pi];
                a.pan_bytes = (uint32_t)(n_cg * w->dev.pan_stride[pi]);
                a.pan_instr = (int32_t)(w->dev.pan_stride[pi] / 1024);
            }
        }
    }
    if (!found) return SL_ERR_UNSUPPORTED;
    return SL_OK;
}

sl_status launch_linear(const sl_packed_weight *w, const int8_t *x, int32_t x_layout, int64_t m, float sx,
                        int32_t kind, float inv_so, void *y, int32_t y_layout, void *stream)
{
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    if (dev != w->dev.device) {
        set_error("handle was packed on device %d, current device is %d", w->dev.device, dev);
        return SL_ERR_INVALID_ARG;
    }
    const TileImage &ti = w->tiles;
    LinearArgs a;
    a.n = w->n_out;
    a.k = w->k_in;
    a.main = w->dev.main;
    a.ovf = w->dev.ovf;
    a.main_bytes = (uint32_t)ti.main.size();
    a.ovf_bytes = (uint32_t)ti.ovf.size();
    a.w_scale = w->dev.w_scale;
    a.bias = w->dev.bias;
    a.sx = sx;
    a.inv_so = inv_so;
    a.n_tiles = ti.n_tiles;
    a.n_win = ti.n_win;
    a.om = nullptr;
    a.pan = nullptr;
    a.pan_bytes = 0;
    a.pan_instr = 0;
    a.n_slices = 0;
    a.slice_groups = 0;
    a.kw = 0;
    hipStream_t s = static_cast<hipStream_t>(stream);

    // (host stack only: the step table is copied out of a fixed-size cache)
    GeluArg ga;
    int32_t run_kind = kind;
    if (kind == SL_EPI_I8_GELU) {
        GeluTable tab;
        if (gelu_table(inv_so, &tab)) {
            ga.hinv = tab.hinv;
            ga.off = tab.off;
            ga.nc = tab.nc;
            ga.pad = 0;
            memcpy(ga.cell, tab.cell, sizeof(ga.cell));
        } else {
            run_kind = kEpiI8GeluErf;
        }
    }
    const bool xt = x_layout == SL_LAYOUT_T16X32, yt = y_layout == SL_LAYOUT_T16X32;
    a.x_cb = (w->k_in + 31) / 32;
    a.y_cb = (w->n_out + 31) / 32;
    // Token rows go through 32-bit buffer offsets: launch at most
    // kMaxBufferBytes of X at a time (a multiple of every workgroup's tokens).
    const int64_t out_bytes = (kind == SL_EPI_I8 || kind == SL_EPI_I8_GELU) ? 1 : 4;
    const int64_t x_token_bytes = xt ? (int64_t)a.x_cb * 32 : w->k_in;
    const int64_t chunk = std::max<int64_t>(256, kMaxBufferBytes / std::max<int64_t>(x_token_bytes, 1) / 256 * 256);
    for (int64_t t0 = 0; t0 < m; t0 += chunk) {
        a.x = x + t0 * x_token_bytes;
        a.y = static_cast<char *>(y) + (yt ? t0 / 16 * a.y_cb * 512 : t0 * w->n_out * out_bytes);
        a.m = std::min(chunk, m - t0);
        const bool vec = xt || ((w->k_in % 16 == 0) && ((reinterpret_cast<uintptr_t>(a.x) & 15) == 0));
        // Aligned or block-layout rows: the weight-stationary kernel where it
        // pays -- a short reduction (at most kPanelMaxWin windows), and a
        // widening layer (N > K: many channel groups share each token row),
        // or slices of at least four token groups per wave (the panel filled
        // once is used for many tokens), or work items of the other kernel
        // that would not make one round of the CUs keeping most of them
        // busy -- with the shape the cost model picks; else the
        // direct-operand kernel (block-layout input, or
        // block-layout output from aligned rows) or the staged kernel
        // (row-major input and output). SL_PATH=panel|direct|staged forces a
        // kernel (tests, tuning; panel falls back when no panel fits).
        // Before all of them, few tokens (at most kSplitAutoItems work items
        // of the split-reduction kernel, about five per compute unit) go to
        // that kernel (SL_PATH=split forces it): there the other kernels'
        // work items would not fill the chip and each walks its whole
        // reduction in series.
        const char *path = env_cfg().path;
        const bool force_split = strcmp(path, "split") == 0;
        const int split_wpw = split_windows_per_wave(ti.n_win);
        const int64_t split_items =
            (a.m + 16 * kSplitSt - 1) / (16 * kSplitSt) * ((ti.n_tiles + kSplitNt - 1) / kSplitNt);
        if (vec && (force_split || (!*path && split_items <= kSplitAutoItems)) && split_wpw > 0) {
            a.n_cgroups = (ti.n_tiles + kSplitNt - 1) / kSplitNt;
            a.om = nullptr;
            a.ovf = w->dev.ovfd;  // (restored below for the other kernels' chunks)
            a.ovf_bytes = w->dev.ovfd_bytes;
            a.n_items = split_items;
            a.kw = (ti.n_win + split_wpw - 1) / split_wpw;
            const sl_status sst = launch_split(a, run_kind == SL_EPI_I8_GELU ? &ga : nullptr, run_kind, xt, yt, s);
            if (sst != SL_OK) return sst;
            set_last_path("split %d,%d kw=%d wpw=%d", kSplitSt, kSplitNt, a.kw, split_wpw);
            a.ovf = w->dev.ovf;
            a.ovf_bytes = (uint32_t)ti.ovf.size();
            continue;
        }
        const bool force_panel = strcmp(path, "panel") == 0;
        const bool auto_path = !*path;
        const bool direct = (xt || (yt && vec) || (vec && strcmp(path, "direct") == 0)) &&
                            !(strcmp(path, "staged") == 0 && !xt && !yt);
        if (vec && (force_panel || (auto_path && ti.n_win <= kPanelMaxWin))) {
            PanelCfg pc{};
            size_t lds = 0;
            sl_status pst = choose_panel_cfg(a, w, run_kind, yt, &pc, &lds);
            if (pst == SL_OK && !force_panel &&
                !(w->n_out > w->k_in || a.slice_groups >= 4 * pc.nwv || !one_full_round(direct, a.m, w)))
                pst = SL_ERR_UNSUPPORTED;
            if (pst == SL_OK) {
                pst = launch_panel(a, run_kind == SL_EPI_I8_GELU ? &ga : nullptr, run_kind, pc, xt, yt, lds, s);
                if (pst != SL_OK) return pst;
                set_last_path("panel %d,%d,%d,%d groups=%d slices=%dx%d lds=%zu", pc.nt, pc.st, pc.nwv, pc.r,
                              a.n_cgroups, a.n_slices, a.slice_groups, lds);
                continue;
            }
            if (pst != SL_ERR_UNSUPPORTED) return pst;
        }
        TileCfg cfg{};
        DirectCfg dcfg{};
        int nt, tm;
        if (direct) {
            dcfg = choose_direct_cfg(a.m, w);
            nt = dcfg.nt;
            tm = dcfg.tm();
        } else {
            cfg = choose_cfg(a.m, w);
            nt = cfg.nt();
            tm = cfg.tm();
        }
        a.n_cgroups = (ti.n_tiles + nt - 1) / nt;
        a.om = nullptr;
        for (int i = 0; i < w->dev.n_om; ++i)
            if (w->dev.om_nt[i] == nt) a.om = w->dev.om[i];
        if (!direct && !a.om) {
            set_error("internal: no overflow table for the chosen workgroup shape");
            return SL_ERR_UNSUPPORTED;
        }
        const int64_t mt = (a.m + tm - 1) / tm;
        a.n_items = mt * a.n_cgroups;
        if (a.n_items > 0x7fffffff) {
            set_error("too many work items for one launch");
            return SL_ERR_UNSUPPORTED;
        }
        sl_status st;
        if (direct) {
            a.ovf = w->dev.ovfd;  // (restored below for the other kernels' chunks)
            a.ovf_bytes = w->dev.ovfd_bytes;
            st = launch_direct(a, run_kind == SL_EPI_I8_GELU ? &ga : nullptr, run_kind, dcfg, xt, yt, s);
            a.ovf = w->dev.ovf;
            a.ovf_bytes = (uint32_t)ti.ovf.size();
            set_last_path("direct %d,%d,%d,%d", dcfg.st, dcfg.nt, dcfg.wm, dcfg.d);
        } else {
            set_last_path("staged %d,%d,%d,%d,%d", cfg.st, cfg.ct, cfg.wm, cfg.wn, cfg.d);
            switch (run_kind) {
            case SL_EPI_ACC_I32: st = launch_vec<SL_EPI_ACC_I32>(a, nullptr, cfg, s, vec, yt); break;
            case SL_EPI_F32: st = launch_vec<SL_EPI_F32>(a, nullptr, cfg, s, vec, yt); break;
            case SL_EPI_F32_GELU: st = launch_vec<SL_EPI_F32_GELU>(a, nullptr, cfg, s, vec, yt); break;
            case SL_EPI_I8: st = launch_vec<SL_EPI_I8>(a, nullptr, cfg, s, vec, yt); break;
            case SL_EPI_I8_GELU: st = launch_vec<SL_EPI_I8_GELU>(a, &ga, cfg, s, vec, yt); break;
            default: st = launch_vec<kEpiI8GeluErf>(a, nullptr, cfg, s, vec, yt); break;
            }
        }
        if (st != SL_OK) return st;
    }
    // the int8 GELU epilogue without a usable step table evaluates erf
    if (run_kind == kEpiI8GeluErf) append_last_path(" gelu=erf");
    return SL_OK;
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

sl_status launch_quantize_t16x32(const float *x, int64_t rows, int32_t cols, float inv_scale, int8_t *q,
                                 void *stream)
{
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int32_t cblocks = (cols + 31) / 32;
    const int64_t n_pieces = (rows + 15) / 16 * cblocks * 32;
    const int64_t blocks = std::min<int64_t>((n_pieces + 255) / 256, 256 * 16);
    const bool vec = cols % 4 == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0;
    if (vec)
        hipLaunchKernelGGL(quantize_t16x32_kernel<true>, dim3((uint32_t)blocks), dim3(256), 0, s, x, rows, cols,
                           cblocks, n_pieces, inv_scale, q);
    else
        hipLaunchKernelGGL(quantize_t16x32_kernel<false>, dim3((uint32_t)blocks), dim3(256), 0, s, x, rows, cols,
                           cblocks, n_pieces, inv_scale, q);
    HIP_TRY(hipGetLastError());
    return SL_OK;
}

}  // namespace sl
