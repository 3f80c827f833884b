// The weight-stationary kernel of the sparse INT8 linear layer (gfx950): for
// token rows that are 16-byte aligned (k_in % 16 == 0) or in SL_LAYOUT_T16X32,
// when a channel group's whole weight panel fits in LDS.
//
// Same method and operand image as the other two kernels (Section "Sparse
// GEMM operators", Figure 1, Algorithm 1: each stored 4x1 block is a value of
// the A operand of the 4:2-sparse int8 matrix instruction, the instruction's
// column indices select the input columns the block mask names, int32
// accumulation, one fused epilogue per output after the whole reduction).
// What differs is the schedule. A workgroup owns one channel group (NT
// 16-channel tiles) and one slice of the tokens. It copies the group's window
// table and whole panel -- every window's NT main operands and NT overflow
// operand slots (zeros where a tile has none in the window), laid out that
// way by the packer -- into LDS once, with no dependent read before the
// copies, then its waves work through the slice's token groups on their own:
// a wave loads its token rows (the B operands) straight into registers,
// R - 1 windows ahead, reads the weight operands from the resident panel a
// few tiles ahead of its matrix instructions, at offsets that follow from
// the window alone, and multiplies every slot, so that no per-tile branch or
// table read sits in the loop (an absent overflow operand is zeros: its
// products are zero). Past the one barrier that follows the panel copy and
// the set-up there is none, so one wave's epilogue overlaps the matrix
// instructions of the others, and the weight image is read from memory once
// per workgroup rather than once per token tile.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "sl_device.h"

namespace sl {

template <int NT, int ST, int NWV>
struct PShape {
    static constexpr int NTH = 64 * NWV;
    static constexpr int TG = 16 * ST;             // tokens per group
    static constexpr int VEC = 2 * NT * kTileN * 4;  // the group's scales sx * sw[n], then its biases
    // per wave: 16 token rows of 32 four-byte outputs (two tiles), padded to
    // 36 words so that neither the writes nor the reads of the transpose meet
    // a bank twice in one pass
    static constexpr int TRW = 36;
    static constexpr int TR = 16 * TRW * 4;
    static_assert(NT <= 32, "an overflow mask has 32 bits");
};

// int32 / fp32 outputs in rows, and int8 outputs in the block layout, go
// through a per-wave LDS transpose
template <int KIND, bool YT, int NT>
constexpr bool panel_transposes()
{
    return NT % 2 == 0 && ((EpiOut<KIND>::kBytes == 4 && KIND != SL_EPI_F32_GELU && !YT) ||
                           (EpiOut<KIND>::kBytes == 1 && YT));
}

// LDS layout: weight scales and biases | GELU step table | per-wave transpose
// areas | window table (n_win + 1 entries of 16 bytes) and panel, as one
// stride of the panel image
template <int KIND, int NT, int ST, int NWV, bool YT>
struct PLds {
    using S = PShape<NT, ST, NWV>;
    static constexpr int kTab = KIND == SL_EPI_I8_GELU ? kGeluLds : 0;
    static constexpr int kTr = panel_transposes<KIND, YT, NT>() ? NWV * S::TR : 0;
    static constexpr int kFixed = S::VEC + kTab + kTr;
    static_assert(kFixed % 16 == 0, "the copies write 16-byte pieces");
    static size_t bytes(uint32_t stride) { return (size_t)kFixed + stride; }
};

// Calls f(std::integral_constant<int, 0>) .. f(std::integral_constant<int, N-1>) in order.
template <int... Us, class F>
__device__ __forceinline__ void static_for_impl(std::integer_sequence<int, Us...>, F &&f)
{
    (f(std::integral_constant<int, Us>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F &&f)
{
    static_for_impl(std::make_integer_sequence<int, N>{}, f);
}

// R: windows of token rows held in registers (R - 1 of them loading while
// one is multiplied)
template <int KIND, int NT, int ST, int NWV, int R, bool XT, bool YT>
__device__ __forceinline__ void panel_body(const LinearArgs &a, const GeluArg *ep)
{
    using S = PShape<NT, ST, NWV>;
    using L = PLds<KIND, NT, ST, NWV, YT>;
    extern __shared__ __attribute__((aligned(16))) int8_t smem[];

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;

    // work: channel group cg, token slice ts; the workgroups of one XCD take
    // consecutive works, which share a token slice
    const int32_t work = (int32_t)xcd_work_index(blockIdx.x, gridDim.x);
    const int32_t ts = work / a.n_cgroups;
    const int32_t cg = work - ts * a.n_cgroups;
    const int32_t tile0 = cg * NT;

    float *const vec = reinterpret_cast<float *>(smem);
    GeluCell *const tab = reinterpret_cast<GeluCell *>(smem + S::VEC);
    int8_t *const trans = smem + S::VEC + L::kTab + wave * S::TR;
    int8_t *const panel = smem + L::kFixed + (a.n_win + 1) * 16;

    // ---- the group's window table and panel: one stride of the panel image,
    // copied global to LDS (no registers) in 1024-byte instructions, wave v
    // issuing instructions v, v + NWV, ...; nothing is read before them, so
    // the copies start at once and land while the set-up runs
    {
        constexpr int kMaxCopies = (int)((kLdsMax / 1024 + NWV - 1) / NWV);
        const __amdgpu_buffer_rsrc_t ir =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.pan, 0, (int)a.pan_bytes, kRsrcWord3);
        const uint32_t src = (uint32_t)cg * (uint32_t)a.pan_instr * 1024u + (uint32_t)lane * 16u;
        int8_t *const dst = smem + L::kFixed;
#pragma unroll
        for (int i = 0; i < kMaxCopies; ++i) {
            const int j = wave + i * NWV;
            if (j < a.pan_instr)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(ir, (lds_void *)(dst + (size_t)j * 1024), 16,
                                                         src + (uint32_t)j * 1024u, 0, 0, 0);
        }
    }

    float hinv = 0.0f, eoff = 0.0f, cmax = 0.0f;  // GELU table parameters (set-up below)


    // ---- token groups of this workgroup's slice, one wave each at a time
    const int64_t mpad = (a.m + 15) / 16 * 16;
    const int64_t slice0 = (int64_t)ts * a.slice_groups * S::TG;
    const int n_groups = (int)std::min<int64_t>(a.slice_groups, (mpad - slice0 + S::TG - 1) / S::TG);
    // this lane's index word: block-row (lane%16)/4, lane group lane/16
    const int iword = ((lane & 15) >> 2) * 4 + (lane >> 4);

    const int64_t xbytes = XT ? mpad / 16 * a.x_cb * 512 : a.m * a.k;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.x, 0, (int)std::min<int64_t>(xbytes, kMaxBufferBytes), kRsrcWord3);
    // Token rows: lane l of subtile s loads features 32*(l/16) .. +31 of the
    // window for token (l % 16) -- the B operand layout. Tokens past m read
    // zeros (out-of-range offsets) or a padding token of the last block; a
    // ragged last window reads bytes past the row (or zeros past the buffer),
    // which meet zero weights.
    auto row_offsets = [&](int64_t t0, uint32_t (&ro)[ST]) {
#pragma unroll
        for (int s = 0; s < ST; ++s) {
            const int64_t r = t0 + s * 16 + (lane & 15);
            if constexpr (XT)
                ro[s] = r < mpad ? (uint32_t)((r >> 4) * a.x_cb * 512) + 512u * (uint32_t)(lane >> 4) +
                                       32u * (uint32_t)(lane & 15)
                                 : kOob;
            else
                ro[s] = r < a.m ? (uint32_t)(r * a.k) + 32u * (uint32_t)(lane >> 4) : kOob;
        }
    };
    // (valid false: every lane reads zeros; the loads are issued all the
    // same, so that the number of loads in flight is the same on every path
    // and the compiler's waits on them stay exact)
    auto load_rows = [&](i32x8 (&bv)[ST], const uint32_t (&ro)[ST], int w, bool valid = true) {
#pragma unroll
        for (int s = 0; s < ST; ++s) {
            const uint32_t off = !valid || ro[s] == kOob ? kOob : ro[s] + (uint32_t)w * (XT ? 4 * 512 : kWin);
            const i32x4 lo = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
            const i32x4 hi = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, off + 16u, 0, 0));
            bv[s] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
    };

    i32x4 acc[NT][ST];
    i32x8 bv[R][ST];
    static_assert(R >= 2, "at least one window loads while another is multiplied");

    // Weight operands in registers, a ring of RS tiles (main operand,
    // overflow slot and their index words) filled LA tiles ahead of the
    // matrix instructions: while tile c of window u is multiplied, tile
    // c + LA of the wave's tile stream is read (of window u, else of window
    // u + 1; past the group's last window that is the first window of the
    // next group, which uses the same panel). A tile's slot is its place in
    // the stream modulo RS; RS divides 2 NT and windows are walked in pairs,
    // so the slot follows from c and the window's parity. Three tiles in
    // flight (NT = 6) instead of two whole windows leave about 90 registers
    // for more waves a SIMD; small tile groups keep a whole window ahead, so
    // that the reads have as many matrix instructions to hide behind.
    constexpr int RS = NT % 3 == 0 ? 3 : (NT <= 2 ? 2 * NT : NT);
    constexpr int LA = RS - 1 < NT ? RS - 1 : NT;
    static_assert((2 * NT) % RS == 0 && LA >= 1, "ring slots follow from the tile and the window's parity");
    struct TOp {
        i32x4 av, ao;
        int ix, io;
    };
    TOp ring[RS];
    auto read_tile = [&](TOp &t, uint32_t base, int c) {
        const int8_t *const wb = panel + base + c * kOpBytes;
        t.av = *reinterpret_cast<const i32x4 *>(wb + lane * 16);
        t.ix = *reinterpret_cast<const int *>(wb + 1024 + iword * 4);
        const int8_t *const oo = panel + base + (NT + c) * kOpBytes;
        t.ao = *reinterpret_cast<const i32x4 *>(oo + lane * 16);
        t.io = *reinterpret_cast<const int *>(oo + 1024 + iword * 4);
    };
    // window u (parity PAR; token rows in ring slot PB, panel bytes cbase;
    // the next window's at nbase)
    auto multiply = [&](auto par, auto pb, uint32_t cbase, uint32_t nbase) {
        constexpr int PAR = decltype(par)::value;
        constexpr int PB = decltype(pb)::value;
        static_for<NT>([&](auto cc) {
            constexpr int C = decltype(cc)::value;
            constexpr int J = C + LA;
            if constexpr (J < NT)
                read_tile(ring[(PAR * NT + J) % RS], cbase, J);
            else
                read_tile(ring[(PAR * NT + J) % RS], nbase, J - NT);
            TOp &t = ring[(PAR * NT + C) % RS];
#pragma unroll
            for (int s = 0; s < ST; ++s)
                acc[C][s] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(t.av, bv[PB][s], acc[C][s], t.ix, 0, 0);
#pragma unroll
            for (int s = 0; s < ST; ++s)
                acc[C][s] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(t.ao, bv[PB][s], acc[C][s], t.io, 0, 0);
            // the four operand reads spread over the tile's matrix
            // instructions, so that a read waiting for room in the LDS queue
            // does not leave the matrix core idle
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);       // one LDS read
                __builtin_amdgcn_sched_group_barrier(0x008, ST / 2, 0);  // matrix instructions
            }
        });
    };

    // accumulator layout: lane l holds rows 4*(l/16)+r (channels of one
    // block-row), column l%16 (token), r = 0..3
    auto scales = [&](int c, float (&s)[4], float (&bb4)[4]) {
        if constexpr (KIND != SL_EPI_ACC_I32) {
            const int lc = c * kTileN + 4 * (lane >> 4);
            const float4 sw = *reinterpret_cast<const float4 *>(vec + lc);
            const float4 bb = *reinterpret_cast<const float4 *>(vec + NT * kTileN + lc);
            s[0] = sw.x;
            s[1] = sw.y;
            s[2] = sw.z;
            s[3] = sw.w;
            bb4[0] = bb.x;
            bb4[1] = bb.y;
            bb4[2] = bb.z;
            bb4[3] = bb.w;
        } else {
            for (int r = 0; r < 4; ++r) s[r] = bb4[r] = 0.0f;
        }
    };
    auto epilogue = [&](int64_t t0) {
        // in the block layout the padding tokens of the last block may be
        // written too
        const int64_t mlim = YT ? mpad : a.m;
        const bool whole = t0 + S::TG <= mlim && (tile0 + NT) * kTileN <= a.n;
        if constexpr (EpiOut<KIND>::kBytes == 1 && YT && panel_transposes<KIND, YT, NT>()) {
            if (whole && tile0 % 2 == 0) {
                // int8 codes in the block layout: a lane holds 4 channels of
                // one token, half of a 32-byte block row; each pair of tiles
                // fills one 512-byte block (16 tokens x 32 channels), which
                // goes through this wave's LDS area so that the store writes
                // the whole block, 8 contiguous bytes a lane
                uint32_t *const tr = reinterpret_cast<uint32_t *>(trans);
                const int wi = (lane & 15) * 8 + (lane >> 4);  // word: token l%16, channels 4(l/16)..
                int8_t *const y8 = static_cast<int8_t *>(a.y);
#pragma unroll
                for (int c = 0; c < NT; c += 2) {
                    float s0[4], b0[4], s1[4], b1[4];
                    scales(c, s0, b0);
                    scales(c + 1, s1, b1);
                    // the GELU kind's table reads for the pair's ST subtiles
                    // are issued together, so that their LDS latency (and
                    // bank conflicts: the cells are data-dependent) is met
                    // once per pair rather than once per two outputs
                    [[maybe_unused]] float gy[ST][2][4];
                    [[maybe_unused]] u32x2 gcell[ST][2][4];
                    if constexpr (KIND == SL_EPI_I8_GELU) {
                        uint32_t ad[ST][2][4];
#pragma unroll
                        for (int st = 0; st < ST; ++st) {
                            gelu_cells(acc[c][st], s0, b0, tab, hinv, eoff, cmax, gy[st][0], ad[st][0]);
                            gelu_cells(acc[c + 1][st], s1, b1, tab, hinv, eoff, cmax, gy[st][1], ad[st][1]);
                        }
#pragma unroll
                        for (int st = 0; st < ST; ++st)
#pragma unroll
                            for (int h = 0; h < 2; ++h)
#pragma unroll
                                for (int r = 0; r < 4; ++r) gcell[st][h][r] = lds_read_u2(ad[st][h][r]);
                    }
#pragma unroll
                    for (int st = 0; st < ST; ++st) {
                        uint32_t v0, v1;
                        if constexpr (KIND == SL_EPI_I8_GELU) {
                            v0 = gelu_codes(gy[st][0], gcell[st][0]);
                            v1 = gelu_codes(gy[st][1], gcell[st][1]);
                        } else {
                            v0 = epilogue_value<KIND>(a, acc[c][st], s0, b0, tab, hinv, eoff, cmax);
                            v1 = epilogue_value<KIND>(a, acc[c + 1][st], s1, b1, tab, hinv, eoff, cmax);
                        }
                        // (a wave's LDS operations take effect in order: the
                        // previous block's read is done before these writes)
                        tr[wi] = v0;
                        tr[wi + 4] = v1;
                        const uint2 r = *reinterpret_cast<const uint2 *>(tr + 2 * lane);
                        int8_t *const p = y8 + t16x32_offset(t0 + st * 16, (tile0 + c) * kTileN, a.y_cb) + 8 * lane;
                        store_nt(p, i32x2{(int)r.x, (int)r.y});
                    }
                }
                return;
            }
        } else if constexpr (panel_transposes<KIND, YT, NT>()) {
            if (whole) {
                // a lane's 16 bytes sit in a different row from its quad
                // neighbours', so each pair of tiles goes through this wave's
                // LDS transpose area; a store then writes 8 tokens x 32
                // channels (128 contiguous bytes a token, 8 lanes a row)
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
        if (whole) {
            // whole group: a uniform base and a lane offset, no bounds checks
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
                    const int64_t uo =
                        YT ? t16x32_offset(t0 + st * 16, ch, a.y_cb) : ((t0 + st * 16) * a.n + ch) * EB;
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

    // The wave's (token group, window) elements form one stream: groups
    // wave, wave + NWV, ... of the slice, each padded to whole turns of the
    // R-window ring, so the u-th window of every group uses ring slot u % R.
    // Before multiplying element e the wave starts loading element e + R - 1
    // (possibly a window of its next group), so the next group's first
    // windows load during the current group's epilogue. The workgroups that
    // share a token slice (one per channel group, on one XCD) would otherwise
    // read the same rows at the same moment: each workgroup visits the
    // slice's groups from its own starting point and each wave walks the
    // windows from its own starting point (int32 sums do not depend on the
    // order).
    const int n_my = n_groups > wave ? (n_groups - wave + NWV - 1) / NWV : 0;
    const int nwp = (a.n_win + R - 1) / R * R;
    const int rot_g = n_groups > 0 ? (int)(((int64_t)cg * 5) % n_groups) : 0;
    const int rot_w = (int)(((int64_t)cg + wave) % a.n_win);
    auto group_t0 = [&](int i) {
        int g = wave + i * NWV + rot_g;
        g = g >= n_groups ? g - n_groups : g;
        return slice0 + (int64_t)g * S::TG;
    };
    auto phys = [&](int u) {
        const int p = u + rot_w;
        return p >= a.n_win ? p - a.n_win : p;
    };
    uint32_t ro[ST], ron[ST];
    // panel byte of the element at window u: NT main operands and NT
    // overflow slots per window
    auto wbase = [&](int u) { return (uint32_t)phys(u) * (uint32_t)(2 * NT * kOpBytes); };
    // the first R - 1 windows of token rows load while the panel copies are
    // in flight, then the set-up; one barrier after all of them, past which
    // table, panel, scales and GELU table are in LDS
    row_offsets(n_my > 0 ? group_t0(0) : slice0, ro);
    static_for<R - 1>([&](auto uc) {
        constexpr int U = decltype(uc)::value;
        load_rows(bv[U], ro, U < a.n_win ? phys(U) : 0, n_my > 0 && U < a.n_win);
    });
    // ---- set-up: scales and biases, GELU table
    static_assert(NT * kTileN <= S::NTH, "one scale and one bias a thread");
    if constexpr (KIND != SL_EPI_ACC_I32) {
        if (tid < NT * kTileN) {
            const int32_t ch = tile0 * kTileN + tid;
            // the dequantisation scale sx * sw[n], one fp32 product as in the definition
            vec[tid] = ch < a.n ? a.sx * a.w_scale[ch] : 0.0f;
            vec[NT * kTileN + tid] = ch < a.n ? a.bias[ch] : 0.0f;
        }
    }
    if constexpr (KIND == SL_EPI_I8_GELU) {
        for (int u = tid; u < ep->nc; u += S::NTH) tab[u] = ep->cell[u];
        hinv = ep->hinv;
        eoff = ep->off;
        cmax = kGeluBase + (float)(ep->nc - 1);
    }
    // every wave's copies (and first token rows) have landed before the barrier
    wait_vmcnt_le<0>();
    __syncthreads();
    if (n_my > 0) {
#pragma unroll
        for (int j = 0; j < LA; ++j) read_tile(ring[j], wbase(0), j);
    }
    static_assert(R % 2 == 0, "ring slots and operand sets alternate together");
    for (int i = 0; i < n_my; ++i) {
        const int64_t t0 = group_t0(i);
        const bool has_next = i + 1 < n_my;
        if (has_next) row_offsets(group_t0(i + 1), ron);
#pragma unroll
        for (int c = 0; c < NT; ++c)
#pragma unroll
            for (int s = 0; s < ST; ++s) acc[c][s] = i32x4{0, 0, 0, 0};
        for (int wb = 0; wb < nwp; wb += R) {
            static_for<R>([&](auto uc) {
                constexpr int U = decltype(uc)::value;
                constexpr int PS = (U + R - 1) % R;
                const int u = wb + U;
                const int pu = u + R - 1;
                const bool in_cur = pu < a.n_win;
                const int pn = pu - nwp;  // window of the next group, if >= 0
                const bool in_next = has_next && pn >= 0 && pn < a.n_win;
                uint32_t rs[ST];
#pragma unroll
                for (int s = 0; s < ST; ++s) rs[s] = in_cur ? ro[s] : ron[s];
                load_rows(bv[PS], rs, in_cur ? phys(pu) : (in_next ? phys(pn) : 0), in_cur || in_next);
                if (u < a.n_win) {
                    // the ring reads ahead into this group's next window,
                    // else the next group's first (a stale read past the
                    // last group)
                    multiply(std::integral_constant<int, U % 2>{}, uc, wbase(u), wbase(u + 1 < a.n_win ? u + 1 : 0));
                }
            });
        }
        // after an odd number of windows the next group's first tiles sit
        // NT slots on; move them to where its first window reads them
        if constexpr (NT % RS != 0) {
            if (a.n_win & 1) {
                static_for<LA>([&](auto tc) {
                    constexpr int T = decltype(tc)::value;
                    ring[T % RS] = ring[(NT + T) % RS];
                });
            }
        }
        epilogue(t0);
        if (has_next) {
#pragma unroll
            for (int s = 0; s < ST; ++s) ro[s] = ron[s];
        }
    }
}

template <int KIND, int NT, int ST, int NWV, int R, bool XT, bool YT>
__global__ __launch_bounds__(64 * NWV) void sparse_linear_panel_kernel(LinearArgs a)
{
    panel_body<KIND, NT, ST, NWV, R, XT, YT>(a, nullptr);
}

template <int NT, int ST, int NWV, int R, bool XT, bool YT>
__global__ __launch_bounds__(64 * NWV) void sparse_linear_panel_gelu_kernel(LinearArgs a, GeluArg ep)
{
    panel_body<SL_EPI_I8_GELU, NT, ST, NWV, R, XT, YT>(a, &ep);
}

template <int KIND, int NT, int ST, int NWV, int R, bool XT, bool YT>
static const void *panel_fn()
{
    if constexpr (KIND == SL_EPI_I8_GELU)
        return reinterpret_cast<const void *>(&sparse_linear_panel_gelu_kernel<NT, ST, NWV, R, XT, YT>);
    else
        return reinterpret_cast<const void *>(&sparse_linear_panel_kernel<KIND, NT, ST, NWV, R, XT, YT>);
}

template <int KIND, int NT, int ST, int NWV, int R, bool XT, bool YT>
static sl_status launch_panel_cfg(const LinearArgs &a, const GeluArg *ep, size_t lds, hipStream_t stream)
{
    using S = PShape<NT, ST, NWV>;
    const void *fn = panel_fn<KIND, NT, ST, NWV, R, XT, YT>();
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
    const int64_t nwg = (int64_t)a.n_cgroups * a.n_slices;
    if constexpr (KIND == SL_EPI_I8_GELU)
        hipLaunchKernelGGL((sparse_linear_panel_gelu_kernel<NT, ST, NWV, R, XT, YT>), dim3((uint32_t)nwg),
                           dim3(S::NTH), lds, stream, a, *ep);
    else
        hipLaunchKernelGGL((sparse_linear_panel_kernel<KIND, NT, ST, NWV, R, XT, YT>), dim3((uint32_t)nwg),
                           dim3(S::NTH), lds, stream, a);
    HIP_TRY(hipGetLastError());
    return SL_OK;
}

// The compiled shapes: F(NT, ST, NWV, R).
#define SL_PANEL_SHAPES(F) \
    F(6, 2, 12, 2)         \
    F(6, 2, 8, 2)          \
    F(4, 2, 8, 2)          \
    F(2, 2, 8, 4)          \
    F(2, 4, 4, 2)

const PanelCfg kPanelCfgs[kNumPanelCfgs] = {
#define SL_PANEL_ENTRY(NT_, ST_, NWV_, R_) {NT_, ST_, NWV_, R_},
    SL_PANEL_SHAPES(SL_PANEL_ENTRY)
#undef SL_PANEL_ENTRY
};

template <int KIND, bool XT, bool YT>
static sl_status launch_panel_kind(const LinearArgs &a, const GeluArg *ep, PanelCfg c, size_t lds,
                                   hipStream_t stream)
{
#define SL_PANEL_CASE(NT_, ST_, NWV_, R_)                                \
    if (c.nt == NT_ && c.st == ST_ && c.nwv == NWV_ && c.r == R_)         \
        return launch_panel_cfg<KIND, NT_, ST_, NWV_, R_, XT, YT>(a, ep, lds, stream);
    SL_PANEL_SHAPES(SL_PANEL_CASE)
#undef SL_PANEL_CASE
    set_error("internal: unknown weight-stationary workgroup shape");
    return SL_ERR_UNSUPPORTED;
}

template <int KIND>
static size_t panel_lds_kind(PanelCfg c, bool yt, uint32_t stride)
{
#define SL_PANEL_LDS(NT_, ST_, NWV_, R_)                                                          \
    if (c.nt == NT_ && c.st == ST_ && c.nwv == NWV_ && c.r == R_)                                 \
        return yt ? PLds<KIND, NT_, ST_, NWV_, true>::bytes(stride)                               \
                  : PLds<KIND, NT_, ST_, NWV_, false>::bytes(stride);
    SL_PANEL_SHAPES(SL_PANEL_LDS)
#undef SL_PANEL_LDS
    return (size_t)-1;
}

size_t panel_lds_bytes(PanelCfg c, int32_t run_kind, bool yt, uint32_t stride)
{
    switch (run_kind) {
    case SL_EPI_ACC_I32: return panel_lds_kind<SL_EPI_ACC_I32>(c, false, stride);
    case SL_EPI_F32: return panel_lds_kind<SL_EPI_F32>(c, false, stride);
    case SL_EPI_F32_GELU: return panel_lds_kind<SL_EPI_F32_GELU>(c, false, stride);
    case SL_EPI_I8: return panel_lds_kind<SL_EPI_I8>(c, yt, stride);
    case SL_EPI_I8_GELU: return panel_lds_kind<SL_EPI_I8_GELU>(c, yt, stride);
    default: return panel_lds_kind<kEpiI8GeluErf>(c, yt, stride);
    }
}

sl_status panel_resident(PanelCfg c, size_t lds, int *out)
{
    const void *fn = nullptr;
    int threads = 0;
#define SL_PANEL_FN(NT_, ST_, NWV_, R_)                                          \
    if (c.nt == NT_ && c.st == ST_ && c.nwv == NWV_ && c.r == R_) {              \
        fn = panel_fn<SL_EPI_F32, NT_, ST_, NWV_, R_, true, false>();            \
        threads = PShape<NT_, ST_, NWV_>::NTH;                                   \
    }
    SL_PANEL_SHAPES(SL_PANEL_FN)
#undef SL_PANEL_FN
    if (!fn) {
        set_error("internal: unknown weight-stationary workgroup shape");
        return SL_ERR_UNSUPPORTED;
    }
    int dev = 0, per_cu = 0, n_cu = 0;
    HIP_TRY(hipGetDevice(&dev));
    HIP_TRY(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax));
    HIP_TRY(hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev));
    HIP_TRY(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, lds));
    *out = per_cu * n_cu;
    return SL_OK;
}

template <int KIND, bool XT>
static sl_status launch_panel_y(const LinearArgs &a, const GeluArg *ep, PanelCfg c, bool yt, size_t lds,
                                hipStream_t stream)
{
    if constexpr (EpiOut<KIND>::kBytes == 1)
        if (yt) return launch_panel_kind<KIND, XT, true>(a, ep, c, lds, stream);
    return launch_panel_kind<KIND, XT, false>(a, ep, c, lds, stream);
}

template <int KIND>
static sl_status launch_panel_x(const LinearArgs &a, const GeluArg *ep, PanelCfg c, bool xt, bool yt, size_t lds,
                                hipStream_t stream)
{
    return xt ? launch_panel_y<KIND, true>(a, ep, c, yt, lds, stream)
              : launch_panel_y<KIND, false>(a, ep, c, yt, lds, stream);
}

sl_status launch_panel(const LinearArgs &a, const GeluArg *ep, int32_t run_kind, PanelCfg c, bool xt, bool yt,
                       size_t lds, hipStream_t stream)
{
    switch (run_kind) {
    case SL_EPI_ACC_I32: return launch_panel_x<SL_EPI_ACC_I32>(a, nullptr, c, xt, yt, lds, stream);
    case SL_EPI_F32: return launch_panel_x<SL_EPI_F32>(a, nullptr, c, xt, yt, lds, stream);
    case SL_EPI_F32_GELU: return launch_panel_x<SL_EPI_F32_GELU>(a, nullptr, c, xt, yt, lds, stream);
    case SL_EPI_I8: return launch_panel_x<SL_EPI_I8>(a, nullptr, c, xt, yt, lds, stream);
    case SL_EPI_I8_GELU: return launch_panel_x<SL_EPI_I8_GELU>(a, ep, c, xt, yt, lds, stream);
    default: return launch_panel_x<kEpiI8GeluErf>(a, nullptr, c, xt, yt, lds, stream);
    }
}

}  // namespace sl
