// The direct-operand kernel of the sparse INT8 linear layer (gfx950): for
// token rows that are 16-byte aligned (k_in % 16 == 0).
//
// Same method and operand image as the staged kernel (Section "Sparse GEMM
// operators", Figure 1, Algorithm 1: the stored 4x1 blocks are one operand of
// the 4:2-sparse int8 matrix instruction, the input columns the weight's mask
// names are selected by the instruction's column indices, int32 accumulation,
// one fused epilogue per output). What differs is where the dense operand
// comes from. Each compute wave owns ST 16-token subtiles and all NT channel
// tiles of the workgroup, so no two waves use the same token rows: a wave
// loads its B operands (32 bytes of one token row per lane) straight from
// memory into registers, two windows ahead, and only the weight operands
// pass through LDS, where all compute waves share them. That halves the LDS
// traffic of a window and leaves LDS bandwidth to the weight operands.
//
// Copy waves stream each window's weight operands into a ring of D LDS
// buffers: the NT main operands and the NT overflow operand slots, both read
// at the same offsets from the main image and from the dense overflow image
// (zeros where a tile has no overflow operand). No table lies on the way to
// a copy's address, so the first element's copies start at kernel entry, and
// every window takes the same number of copies, which keeps the waits that
// count them constant. Work items (token tile x channel group) are spread
// over a persistent grid.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "sl_device.h"

namespace sl {

// Workgroup shape: WM compute waves along the tokens, each with ST 16-token
// subtiles x all NT 16-channel tiles; as many copy waves; D windows in flight.
// One window's buffer: NT main operands, then NT overflow operand slots (one
// per tile, zeros where the tile has none); each region is padded to whole
// 64-lane copies per copy wave.
template <int ST, int NT, int WM, int D>
struct DShape {
    static constexpr int NW = WM;
    static constexpr int NTH = 64 * NW;                          // lanes of the compute (and of the copy) waves
    static constexpr int NTHG = 2 * NTH;                         // threads per workgroup
    static constexpr int TM = 16 * ST * WM;                      // tokens per work item
    static constexpr int CA = (NT * kOpPieces + NTH - 1) / NTH;  // copies per copy wave per region
    static constexpr int AB = CA * NTH * 16;
    static constexpr int COPIES = 2 * CA;  // per copy wave per window: main, overflow
    static constexpr int BUF = 2 * AB;
    static constexpr int LDS = D * BUF;
    static constexpr int VEC = 2 * NT * kTileN * 4;  // per compute wave: weight scales, then biases
    // per compute wave: 16 token rows of 32 four-byte outputs (two tiles),
    // padded to 36 words so that neither the writes nor the reads of the
    // transpose meet a bank twice in one pass
    static constexpr int TRW = 36;
    static constexpr int TR = 16 * TRW * 4;
    static_assert(NT <= 32, "an overflow mask has 32 bits");
};

// XT: x in SL_LAYOUT_T16X32 (else row-major, 16-byte aligned rows); YT: y in
// SL_LAYOUT_T16X32 (int8 kinds).
template <int KIND, int ST, int NT, int WM, int D, bool XT, bool YT>
__device__ __forceinline__ void direct_body(const LinearArgs &a, const GeluArg *ep)
{
    using S = DShape<ST, NT, WM, D>;
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    // waves 0..NW-1 load the token rows and run the matrix instructions;
    // waves NW..2NW-1 only copy weight operands
    const bool copier = wave >= S::NW;
    const int pw = copier ? wave - S::NW : 0;

    const int32_t G = (int32_t)gridDim.x;
    const int32_t slot = (int32_t)xcd_work_index(blockIdx.x, G);
    const int n_my = (int)((a.n_items - slot + G - 1) / G);  // >= 1: the grid is at most n_items
    const int64_t steps = (int64_t)n_my * a.n_win;
    const ItemIter first = ItemIter::start(slot, G, a.n_cgroups, a.n_win);
    auto phys = [&](const ItemIter &it, int w) {
        const int p = w + it.rot;
        return p >= a.n_win ? p - a.n_win : p;
    };

    // LDS: the ring, the GELU table, the compute waves' scales and biases
    GeluCell *tab = reinterpret_cast<GeluCell *>(smem + S::LDS);
    constexpr int kTabBytes = KIND == SL_EPI_I8_GELU ? kGeluLds : 0;
    float hinv = 0.0f, eoff = 0.0f, cmax = 0.0f;
    if constexpr (KIND == SL_EPI_I8_GELU) {
        for (int u = copier ? ep->nc : tid; u < ep->nc; u += S::NTH) tab[u] = ep->cell[u];
        hinv = ep->hinv;
        eoff = ep->off;
        cmax = kGeluBase + (float)(ep->nc - 1);
    }

    // Pipeline over the (item, window) elements, one barrier per element. In
    // step e the copy waves wait until element e+1 has landed, pass the
    // barrier and start the copies of element e+D into the buffer of element
    // e; the compute waves pass the barrier, read element e+1's weight
    // operands into one register set while element e's matrix instructions
    // run from the other, start the token-row loads of element e+2, and wait
    // for their LDS reads before the next barrier.
    static_assert(D >= 3, "the pipeline reads one element ahead of the one it multiplies");
    static_assert((D - 1) * S::COPIES < 64, "outstanding copies must fit the 6-bit vector-memory counter");

    if (copier) {
        const __amdgpu_buffer_rsrc_t mr =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.main, 0, (int)a.main_bytes, kRsrcWord3);
        const __amdgpu_buffer_rsrc_t orc =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.ovf, 0, (int)a.ovf_bytes, kRsrcWord3);
        const uint32_t wstride = (uint32_t)a.n_tiles * kOpBytes;  // main image bytes per window
        // this lane's piece (tile, 16-byte piece) of each operand-region copy
        int32_t atile[S::CA], apiece16[S::CA];
#pragma unroll
        for (int i = 0; i < S::CA; ++i) {
            const int piece = (i * S::NW + pw) * 64 + lane;
            atile[i] = piece / kOpPieces;
            apiece16[i] = (piece - atile[i] * kOpPieces) * 16;
        }

        // element cursor (item ic, the kc-th of this workgroup; window wc);
        // past the last element it repeats the last one
        ItemIter ic = first;
        int kc = 0, wc = 0;
        auto cur_w = [&]() { return phys(ic, kc < n_my ? wc : a.n_win - 1); };
        uint32_t aoff[S::CA];
        auto item_offsets = [&]() {
            const int32_t tile0 = ic.cg * NT;
            const int32_t ntl = min(NT, a.n_tiles - tile0);
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

        // Copy k (0 <= k < COPIES) of the cursor's element (physical window
        // w) into ring buffer bi: main operands, then overflow slots.
        auto copy = [&](int k, int w, int bi) {
            int8_t *b = smem + bi * S::BUF;
            const uint32_t wo = (uint32_t)w * wstride;
            if (k < S::CA)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(mr, (lds_void *)(b + (k * S::NW + pw) * 1024), 16, aoff[k],
                                                         wo, 0, 0);
            else
                __builtin_amdgcn_raw_ptr_buffer_load_lds(orc, (lds_void *)(b + S::AB + ((k - S::CA) * S::NW + pw) * 1024),
                                                         16, aoff[k - S::CA], wo, 0, 0);
        };

        // Prologue: the copies of elements 0..D-1, element by element; a bare
        // barrier (A) publishes the epilogue table the compute waves filled;
        // once element 0 has landed a second barrier (B) publishes it.
#pragma unroll
        for (int d = 0; d < D; ++d) {
            const int w = cur_w();
#pragma unroll
            for (int k = 0; k < S::COPIES; ++k) copy(k, w, d);
            advance();
        }
        __builtin_amdgcn_s_barrier();  // (A)
        asm volatile("" ::: "memory");
        wait_vmcnt_le<(D - 1) * S::COPIES>();  // element 0 landed
        __builtin_amdgcn_s_barrier();          // (B)
        asm volatile("" ::: "memory");

        // step e: wait until element e+1 has landed (the copies issued after
        // it are those of the D-2 elements that follow it), then copy element
        // e+D into the buffer of element e
        auto cstep = [&](int64_t e, int u) {
            if (e + 1 < steps) wait_vmcnt_le<(D - 2) * S::COPIES>();
            // a bare barrier: __syncthreads() would also wait for the later
            // elements' copies still in flight
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            const int w = cur_w();
#pragma unroll
            for (int k = 0; k < S::COPIES; ++k) copy(k, w, u);
            advance();
        };
        int64_t e = 0;
        for (; e + D <= steps; e += D) {
#pragma unroll
            for (int u = 0; u < D; ++u) cstep(e + u, u);
        }
#pragma unroll
        for (int u = 0; u < D; ++u)
            if (e + u < steps) cstep(e + u, u);
        __builtin_amdgcn_s_waitcnt(0);  // no copy may land after the workgroup ends
        return;
    }
    __builtin_amdgcn_s_waitcnt(0);  // the epilogue table's LDS stores are done
    __builtin_amdgcn_s_barrier();   // (A)
    asm volatile("" ::: "memory");

    // ---- compute waves
    const int wm = wave;
    // this lane's index word: block-row (lane%16)/4, lane group lane/16
    const int iword = ((lane & 15) >> 2) * 4 + (lane >> 4);

    // Token rows: lane l of subtile s loads features 32*(l/16) .. +31 of its
    // window for token (l % 16) -- the B operand layout. Row-major: 32 bytes
    // of the token's row; block layout: 32 bytes of the token's row in block
    // 4w + l/16, so each group of 4 lanes reads one cache line. Tokens past m
    // read zeros (out-of-range offsets) or a padding token of the last block;
    // a ragged last window reads bytes past the row (or zeros past the
    // buffer), which meet zero weights.
    const int64_t xbytes = XT ? (a.m + 15) / 16 * a.x_cb * 512 : a.m * a.k;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.x, 0, (int)min<int64_t>(xbytes, kMaxBufferBytes), kRsrcWord3);
    auto row_offsets = [&](const ItemIter &it, uint32_t (&ro)[ST]) {
#pragma unroll
        for (int s = 0; s < ST; ++s) {
            const int64_t r = (int64_t)it.mt * S::TM + wm * ST * 16 + s * 16 + (lane & 15);
            if constexpr (XT)
                ro[s] = r < (a.m + 15) / 16 * 16 ? (uint32_t)((r >> 4) * a.x_cb * 512) + 512u * (uint32_t)(lane >> 4) +
                                                       32u * (uint32_t)(lane & 15)
                                                 : kOob;
            else
                ro[s] = r < a.m ? (uint32_t)(r * a.k) + 32u * (uint32_t)(lane >> 4) : kOob;
        }
    };
    auto load_rows = [&](i32x8 (&bv)[ST], const uint32_t (&ro)[ST], int w) {
#pragma unroll
        for (int s = 0; s < ST; ++s) {
            const uint32_t off = ro[s] + (uint32_t)w * (XT ? 4 * 512 : kWin);
            const i32x4 lo = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
            const i32x4 hi = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off + 16u, 0, 0));
            bv[s] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
    };

    // Weight operands of one element in registers: main and overflow A
    // operands of every tile with their index words (an absent overflow
    // operand is zeros: its products are zero). Two sets alternate (steps e,
    // e+1), for the token rows too: element e+1's rows load at the start of
    // step e, into the set whose matrix instructions (step e-1's) have been
    // issued before the barrier, so the loads do not wait for them.
    struct Ops {
        i32x4 av[NT], ao[NT];
        int ix[NT], io[NT];
    };
    Ops ops[2];
    i32x8 bv[2][ST];
    auto read_ops = [&](Ops &r, const int8_t *b) {
#pragma unroll
        for (int c = 0; c < NT; ++c) {
            const int8_t *op = b + c * kOpBytes;
            r.av[c] = *reinterpret_cast<const i32x4 *>(op + lane * 16);
            r.ix[c] = *reinterpret_cast<const int *>(op + 1024 + iword * 4);
            const int8_t *oo = b + S::AB + c * kOpBytes;
            r.ao[c] = *reinterpret_cast<const i32x4 *>(oo + lane * 16);
            r.io[c] = *reinterpret_cast<const int *>(oo + 1024 + iword * 4);
        }
    };

    // the item's weight scales and biases, one copy each into this wave's
    // LDS area (NT*4 lanes of 16 bytes); the epilogue waits for them
    float *vec = reinterpret_cast<float *>(smem + S::LDS + kTabBytes + wave * S::VEC);
    int8_t *const trans = smem + S::LDS + kTabBytes + S::NW * S::VEC + wave * S::TR;
    auto fetch_vec = [&](const ItemIter &it) {
        if constexpr (KIND != SL_EPI_ACC_I32) {
            const __amdgpu_buffer_rsrc_t sr =
                __builtin_amdgcn_make_buffer_rsrc((void *)a.w_scale, 0, a.n * 4, kRsrcWord3);
            const __amdgpu_buffer_rsrc_t br = __builtin_amdgcn_make_buffer_rsrc((void *)a.bias, 0, a.n * 4, kRsrcWord3);
            if (lane < NT * 4) {
                const uint32_t off = (uint32_t)((it.cg * NT * kTileN + lane * 4) * 4);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(sr, (lds_void *)vec, 16, off, 0, 0, 0);
                __builtin_amdgcn_raw_ptr_buffer_load_lds(br, (lds_void *)(vec + NT * kTileN), 16, off, 0, 0, 0);
            }
        }
    };

    i32x4 acc[NT][ST];
    auto clear_acc = [&]() {
#pragma unroll
        for (int c = 0; c < NT; ++c)
#pragma unroll
            for (int s = 0; s < ST; ++s) acc[c][s] = i32x4{0, 0, 0, 0};
    };
    // accumulator layout: lane l holds rows 4*(l/16)+r (channels of one
    // block-row), column l%16 (token), r = 0..3
    auto epilogue = [&](const ItemIter &it) {
        __builtin_amdgcn_s_waitcnt(0);  // this wave's scale and bias copies
        const int64_t t0 = (int64_t)it.mt * S::TM + wm * ST * 16;  // this wave's first token
        const int32_t tile0 = it.cg * NT;
        auto scales = [&](int c, float (&s)[4], float (&bb4)[4]) {
            if constexpr (KIND != SL_EPI_ACC_I32) {
                const int lc = c * kTileN + 4 * (lane >> 4);
                const float4 sw = *reinterpret_cast<const float4 *>(vec + lc);
                const float4 bb = *reinterpret_cast<const float4 *>(vec + NT * kTileN + lc);
                s[0] = a.sx * sw.x;
                s[1] = a.sx * sw.y;
                s[2] = a.sx * sw.z;
                s[3] = a.sx * sw.w;
                bb4[0] = bb.x;
                bb4[1] = bb.y;
                bb4[2] = bb.z;
                bb4[3] = bb.w;
            } else {
                for (int r = 0; r < 4; ++r) s[r] = bb4[r] = 0.0f;
            }
        };
        // in the block layout the padding tokens of the last block may be
        // written too
        const int64_t mlim = YT ? (a.m + 15) / 16 * 16 : a.m;
        if constexpr (EpiOut<KIND>::kBytes == 4 && KIND != SL_EPI_F32_GELU && !YT && NT % 2 == 0) {
            if (t0 + ST * 16 <= mlim && (tile0 + NT) * kTileN <= a.n) {
                // Whole tile, int32 or fp32 outputs in rows (the fp32 GELU kind
                // keeps the direct stores: two tiles of its temporaries at once
                // would spill): a lane's 16 bytes sit in
                // a different row from its quad neighbours', so each pair of
                // tiles goes through this wave's LDS transpose area. A store
                // then writes 8 tokens x 32 channels (128 contiguous bytes a
                // token, 8 lanes a row).
                int32_t *const tr = reinterpret_cast<int32_t *>(trans);
                const int wi = (lane & 15) * S::TRW + 4 * (lane >> 4);  // write: token l%16, channels 4(l/16)..
                const int ri = (lane >> 3) * S::TRW + 4 * (lane & 7);   // read: token l/8 (+8), channels 4(l%8)..
                int8_t *const y8 = static_cast<int8_t *>(a.y);
#pragma unroll
                for (int c = 0; c < NT; c += 2) {
                    float s0[4], b0[4], s1[4], b1[4];
                    scales(c, s0, b0);
                    scales(c + 1, s1, b1);
#pragma unroll
                    for (int st = 0; st < ST; ++st) {
                        const i32x4 v0 = __builtin_bit_cast(
                            i32x4, epilogue_value<KIND>(a, acc[c][st], s0, b0, tab, hinv, eoff, cmax));
                        const i32x4 v1 = __builtin_bit_cast(
                            i32x4, epilogue_value<KIND>(a, acc[c + 1][st], s1, b1, tab, hinv, eoff, cmax));
                        // (a wave's LDS operations take effect in order: the
                        // previous pair's reads are done before these writes)
                        *reinterpret_cast<i32x4 *>(tr + wi) = v0;
                        *reinterpret_cast<i32x4 *>(tr + wi + 16) = v1;
                        const i32x4 r0 = *reinterpret_cast<const i32x4 *>(tr + ri);
                        const i32x4 r1 = *reinterpret_cast<const i32x4 *>(tr + ri + 8 * S::TRW);
                        const int64_t row = t0 + st * 16 + (lane >> 3);
                        int8_t *const p = y8 + (row * a.n + (tile0 + c) * kTileN + 4 * (lane & 7)) * 4;
                        store_nt(p, r0);
                        store_nt(p + (int64_t)8 * a.n * 4, r1);
                    }
                }
                return;
            }
        }
        if (t0 + ST * 16 <= mlim && (tile0 + NT) * kTileN <= a.n) {
            // whole tile: a uniform base and a lane offset, no bounds checks
            constexpr int EB = EpiOut<KIND>::kBytes;
            int8_t *const y8 = static_cast<int8_t *>(a.y);
            const uint32_t lo = YT ? (uint32_t)(32 * (lane & 15) + 4 * (lane >> 4))
                                   : (uint32_t)(((lane & 15) * a.n + 4 * (lane >> 4)) * EB);
#pragma unroll
            for (int c = 0; c < NT; ++c) {
                float s[4], bb4[4];
                scales(c, s, bb4);
#pragma unroll
                for (int st = 0; st < ST; ++st) {
                    const int32_t ch = (tile0 + c) * kTileN;
                    const int64_t uo = YT ? t16x32_offset(t0 + st * 16, ch, a.y_cb)
                                          : ((t0 + st * 16) * a.n + ch) * EB;
                    store_nt(y8 + uo + lo, epilogue_value<KIND>(a, acc[c][st], s, bb4, tab, hinv, eoff, cmax));
                }
            }
        } else {
#pragma unroll
            for (int c = 0; c < NT; ++c) {
                const int32_t t = tile0 + c;
                if (t >= a.n_tiles) break;
                const int32_t ch0 = t * kTileN + 4 * (lane >> 4);
                if (ch0 >= a.n) continue;  // block-rows past n_out in the last tile
                float s[4], bb4[4];
                scales(c, s, bb4);
#pragma unroll
                for (int st = 0; st < ST; ++st)
                    epilogue_store<KIND, YT>(a, acc[c][st], t0 + st * 16 + (lane & 15), ch0, s, bb4, tab, hinv,
                                             eoff, cmax);
            }
        }
    };

    // element cursor of the token-row loads (element e+1 in step e: item ib,
    // window wb); sl: element e's ring buffer
    ItemIter ib = first;
    int kb = 0, wb = 0;
    uint32_t rob[ST];
    row_offsets(ib, rob);
    auto load_next_rows = [&](i32x8 (&dst)[ST]) {
        load_rows(dst, rob, phys(ib, kb < n_my ? wb : a.n_win - 1));
        if (++wb == a.n_win) {
            wb = 0;
            if (++kb < n_my) {
                ib.next();
                row_offsets(ib, rob);
            }
        }
    };
    int sl = 0;
    // step of element e with its weight operands and token rows in set PA
    // (e % 2)
    auto step = [&](auto pa) {
        constexpr int PA = decltype(pa)::value;
        Ops &cur = ops[PA];
        Ops &nxt = ops[PA ^ 1];
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        load_next_rows(bv[PA ^ 1]);  // element e+1's token rows
        sl = sl + 1 == D ? 0 : sl + 1;
        // element e+1's operand reads, one before each matrix instruction of
        // element e, so that a read waiting for room in the LDS queue does not
        // leave the matrix core idle. (The last step reads a stale buffer:
        // harmless.) Products of tiles past the item's last tile land in
        // accumulators that are never stored.
        read_ops(nxt, smem + sl * S::BUF);
        // (all main products first, then the overflow ones: an instruction
        // never waits for the result of the one just before it)
#pragma unroll
        for (int c = 0; c < NT; ++c)
#pragma unroll
            for (int s = 0; s < ST; ++s)
                acc[c][s] =
                    __builtin_amdgcn_smfmac_i32_16x16x128_i8(cur.av[c], bv[PA][s], acc[c][s], cur.ix[c], 0, 0);
#pragma unroll
        for (int c = 0; c < NT; ++c)
#pragma unroll
            for (int s = 0; s < ST; ++s)
                acc[c][s] =
                    __builtin_amdgcn_smfmac_i32_16x16x128_i8(cur.ao[c], bv[PA][s], acc[c][s], cur.io[c], 0, 0);
#pragma unroll
        for (int v = 0; v < 4 * NT; ++v) {
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one matrix instruction
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * NT * ST, 0);  // the remaining matrix instructions
        // element e+1's buffer is refilled after the next barrier: its reads
        // must be done by then
        wait_lgkm0();
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;

    ItemIter it = first;
    clear_acc();
    fetch_vec(it);
    load_next_rows(bv[0]);
    __builtin_amdgcn_s_barrier();  // (B): element 0 has landed
    asm volatile("" ::: "memory");
    read_ops(ops[0], smem);
    wait_lgkm0();  // element 0's buffer is refilled after the next barrier
    // Each item starts with its first element in set 0; after an odd number
    // of windows the next element's operands are moved there from set 1.
    for (int k = 0; k < n_my; ++k) {
        int w = 0;
        for (; w + 2 <= a.n_win; w += 2) {
            step(I0{});
            step(I1{});
        }
        if (w < a.n_win) step(I0{});
        epilogue(it);  // (waits for every load: the moves below read loaded registers)
        if (w < a.n_win) {
            ops[0] = ops[1];
#pragma unroll
            for (int s = 0; s < ST; ++s) bv[0][s] = bv[1][s];
        }
        if (k + 1 < n_my) {
            clear_acc();
            it.next();
            asm volatile("" ::: "memory");  // the epilogue's reads of the scales come first
            fetch_vec(it);
        }
    }
}

template <int KIND, int ST, int NT, int WM, int D, bool XT, bool YT>
__global__ __launch_bounds__(128 * WM) void sparse_linear_direct_kernel(LinearArgs a)
{
    direct_body<KIND, ST, NT, WM, D, XT, YT>(a, nullptr);
}

template <int ST, int NT, int WM, int D, bool XT, bool YT>
__global__ __launch_bounds__(128 * WM) void sparse_linear_direct_gelu_kernel(LinearArgs a, GeluArg ep)
{
    direct_body<SL_EPI_I8_GELU, ST, NT, WM, D, XT, YT>(a, &ep);
}

template <int KIND, int ST, int NT, int WM, int D, bool XT, bool YT>
static sl_status launch_direct_cfg(const LinearArgs &a, const GeluArg *ep, hipStream_t stream)
{
    using S = DShape<ST, NT, WM, D>;
    const void *fn;
    if constexpr (KIND == SL_EPI_I8_GELU)
        fn = reinterpret_cast<const void *>(&sparse_linear_direct_gelu_kernel<ST, NT, WM, D, XT, YT>);
    else
        fn = reinterpret_cast<const void *>(&sparse_linear_direct_kernel<KIND, ST, NT, WM, D, XT, YT>);
    constexpr size_t kTrans = EpiOut<KIND>::kBytes == 4 && KIND != SL_EPI_F32_GELU && !YT ? S::NW * S::TR : 0;
    const size_t lds = (size_t)S::LDS + S::NW * S::VEC + kTrans + (KIND == SL_EPI_I8_GELU ? kGeluLds : 0);
    static_assert(S::LDS + S::NW * (S::VEC + S::TR) + kGeluLds <= kLdsMax, "workgroup shape exceeds LDS");
    static int resident[kMaxDevices] = {};  // per kernel instance and device
    int grid = 0;
    const sl_status st = persistent_grid(fn, S::NTHG, lds, resident, &grid);
    if (st != SL_OK) return st;
    const int64_t nwg = std::min<int64_t>(a.n_items, grid);
    if constexpr (KIND == SL_EPI_I8_GELU)
        hipLaunchKernelGGL((sparse_linear_direct_gelu_kernel<ST, NT, WM, D, XT, YT>), dim3((uint32_t)nwg),
                           dim3(S::NTHG), lds, stream, a, *ep);
    else
        hipLaunchKernelGGL((sparse_linear_direct_kernel<KIND, ST, NT, WM, D, XT, YT>), dim3((uint32_t)nwg),
                           dim3(S::NTHG), lds, stream, a);
    HIP_TRY(hipGetLastError());
    return SL_OK;
}

template <int KIND, bool XT, bool YT>
static sl_status launch_direct_kind(const LinearArgs &a, const GeluArg *ep, DirectCfg c, hipStream_t stream)
{
#define SL_DCFG(A_, B_, C_, D_)                                \
    if (c.st == A_ && c.nt == B_ && c.wm == C_ && c.d == D_) \
        return launch_direct_cfg<KIND, A_, B_, C_, D_, XT, YT>(a, ep, stream);
    SL_DCFG(2, 6, 4, 4)
    SL_DCFG(1, 6, 4, 6)
    SL_DCFG(1, 2, 4, 8)
#undef SL_DCFG
    set_error("internal: unknown direct workgroup shape");
    return SL_ERR_UNSUPPORTED;
}

const DirectCfg kDirectCfgs[kNumDirectCfgs] = {
    {2, 6, 4, 4},  // 128 tokens x 96 channels
    {1, 6, 4, 6},  //  64 tokens x 96 channels
    {1, 2, 4, 8},  //  64 tokens x 32 channels (few work items)
};

template <int KIND, bool XT>
static sl_status launch_direct_y(const LinearArgs &a, const GeluArg *ep, DirectCfg c, bool yt, hipStream_t stream)
{
    if constexpr (EpiOut<KIND>::kBytes == 1)
        if (yt) return launch_direct_kind<KIND, XT, true>(a, ep, c, stream);
    return launch_direct_kind<KIND, XT, false>(a, ep, c, stream);
}

template <int KIND>
static sl_status launch_direct_x(const LinearArgs &a, const GeluArg *ep, DirectCfg c, bool xt, bool yt,
                                 hipStream_t stream)
{
    return xt ? launch_direct_y<KIND, true>(a, ep, c, yt, stream) : launch_direct_y<KIND, false>(a, ep, c, yt, stream);
}

sl_status launch_direct(const LinearArgs &a, const GeluArg *ep, int32_t run_kind, DirectCfg c, bool xt, bool yt,
                        hipStream_t stream)
{
    switch (run_kind) {
    case SL_EPI_ACC_I32: return launch_direct_x<SL_EPI_ACC_I32>(a, nullptr, c, xt, yt, stream);
    case SL_EPI_F32: return launch_direct_x<SL_EPI_F32>(a, nullptr, c, xt, yt, stream);
    case SL_EPI_F32_GELU: return launch_direct_x<SL_EPI_F32_GELU>(a, nullptr, c, xt, yt, stream);
    case SL_EPI_I8: return launch_direct_x<SL_EPI_I8>(a, nullptr, c, xt, yt, stream);
    case SL_EPI_I8_GELU: return launch_direct_x<SL_EPI_I8_GELU>(a, ep, c, xt, yt, stream);
    default: return launch_direct_x<kEpiI8GeluErf>(a, nullptr, c, xt, yt, stream);
    }
}

}  // namespace sl
