// Host packer: dense int8 weight -> canonical 4x1 BSR -> GPU tile image.
//
// Section "Sparse GEMM operators": the sparse weight is stored compressed and
// its mask (the column index of every stored block) drives the
// reorganisation of the input. Appendix "Block-wise structured sparsity": the
// blocks are 1-D, 4 consecutive output rows at one input column.
//
// The GPU image regroups 4 block-rows into a 16-channel tile, the A operand of
// the 4:2-sparse matrix-core instruction v_smfmac_i32_16x16x128_i8. In each
// 128-column window, a block-row's stored blocks fall into aligned groups of 4
// columns; the instruction takes at most 2 values per row and group, selected
// by 2-bit column indices -- the block mask becomes the instruction's sparsity
// index, and the hardware picks the matching input columns, which is the
// paper's mask-driven reorganisation of the input. The first two stored blocks
// of every (block-row, group) go to the window's main entry; the rare third
// and fourth go to an overflow entry on the same window. All 4 rows of a block
// share its columns, so each stored block is 4 values with one index.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <new>

#include "sl_internal.h"

namespace sl {

sl_status validate_weight_args(const int8_t *w, int32_t n_out, int32_t k_in, int32_t bh, int32_t bw,
                               const float *w_scale, const float *bias)
{
    if (!w || !w_scale) {
        set_error("w_host and w_scale_host must not be NULL");
        return SL_ERR_INVALID_ARG;
    }
    if (bh != 4 || bw != 1) {
        set_error("only 4x1 blocks (4 consecutive output rows, 1 input column) are supported");
        return SL_ERR_INVALID_ARG;
    }
    if (n_out < 4 || n_out % 4 != 0) {
        set_error("n_out must be a positive multiple of 4 (no padding of partial blocks)");
        return SL_ERR_SHAPE;
    }
    if (k_in < 1 || k_in > 65535) {
        set_error("k_in must be in [1, 65535] (16-bit column index)");
        return SL_ERR_SHAPE;
    }
    for (int32_t n = 0; n < n_out; ++n) {
        if (!(isfinite(w_scale[n]) && w_scale[n] > 0.0f)) {
            set_error("w_scale must be finite and > 0 (channel %d)", (int)n);
            return SL_ERR_INVALID_ARG;
        }
        if (bias && !isfinite(bias[n])) {
            set_error("bias must be finite (channel %d)", (int)n);
            return SL_ERR_INVALID_ARG;
        }
    }
    return SL_OK;
}

static sl_status build_bsr(const int8_t *w, int32_t n_out, int32_t k_in, sl_packed_weight *p)
{
    const int32_t nbr = n_out / 4;
    p->row_ptr.assign(nbr + 1, 0);
    p->col.clear();
    p->vals.clear();
    for (int32_t g = 0; g < nbr; ++g) {
        const int8_t *r0 = w + (int64_t)(4 * g) * k_in;
        for (int32_t k = 0; k < k_in; ++k) {
            int8_t v0 = r0[k], v1 = r0[k_in + k], v2 = r0[2 * (int64_t)k_in + k], v3 = r0[3 * (int64_t)k_in + k];
            if (v0 | v1 | v2 | v3) {
                p->col.push_back((uint16_t)k);
                p->vals.push_back(v0);
                p->vals.push_back(v1);
                p->vals.push_back(v2);
                p->vals.push_back(v3);
            }
        }
        p->row_ptr[g + 1] = (uint32_t)p->col.size();
    }
    p->nnzb = (int64_t)p->col.size();
    return SL_OK;
}

// Group g of a window -> (lane group q, value pair t) with entry_group(q, t) == g.
static void group_slot(int g, int *q, int *t)
{
    for (int qq = 0; qq < 4; ++qq)
        for (int tt = 0; tt < 8; ++tt)
            if (entry_group(qq, tt) == g) {
                *q = qq;
                *t = tt;
                return;
            }
}

// Default index nibble of a pair with no stored value: positions (0, 1).
constexpr uint32_t kIdleIdx = 0x44444444u;

// The instruction's value pair for the n (1 or 2) stored blocks eg[0..n-1] of
// one (block-row, aligned 4-column group): positions ascending and distinct;
// a lone block is paired with an unused position that holds no value
// (blk = UINT32_MAX).
static void make_pair(const sl_packed_weight *p, const uint32_t *eg, int n, int pos[2], uint32_t blk[2])
{
    blk[0] = blk[1] = UINT32_MAX;
    pos[0] = p->col[eg[0]] % 4;
    blk[0] = eg[0];
    if (n == 2) {
        pos[1] = p->col[eg[1]] % 4;
        blk[1] = eg[1];
    } else if (pos[0] < 3) {
        pos[1] = 3;
    } else {
        pos[0] = 2;
        pos[1] = 3;
        blk[1] = blk[0];
        blk[0] = UINT32_MAX;
    }
}

static sl_status build_tiles(sl_packed_weight *p)
{
    TileImage &ti = p->tiles;
    const int32_t nbr = p->n_out / 4;
    const int32_t k_in = p->k_in;
    ti.n_tiles = (p->n_out + kTileN - 1) / kTileN;
    ti.n_win = (k_in + kWin - 1) / kWin;
    const size_t pstride = (size_t)ti.n_tiles + 1;
    ti.main.assign((size_t)ti.n_win * ti.n_tiles * kOpBytes, 0);
    ti.ovf.clear();
    ti.ovf_ptr.assign((size_t)ti.n_win * pstride, 0);
    ti.n_entries = 0;
    ti.n_overflow = 0;

    int gq[32], gt[32];
    for (int g = 0; g < 32; ++g) group_slot(g, &gq[g], &gt[g]);

    std::vector<uint32_t> cur(p->row_ptr.begin(), p->row_ptr.end() - 1);  // per block-row cursor
    int8_t op[2][kOpBytes];
    uint32_t n_ovf = 0;
    for (int32_t w = 0; w < ti.n_win; ++w) {
        const int32_t wbeg = w * kWin, wend = std::min(k_in, wbeg + kWin);
        for (int32_t t = 0; t < ti.n_tiles; ++t) {
            ti.ovf_ptr[(size_t)w * pstride + t] = n_ovf;
            memset(op, 0, sizeof(op));
            uint32_t idx[2][16];
            for (int sl = 0; sl < 2; ++sl)
                for (int i = 0; i < 16; ++i) idx[sl][i] = kIdleIdx;
            bool used[2] = {false, false};
            const int32_t g0 = 4 * t, g1 = std::min(4 * t + 4, nbr);
            for (int32_t g = g0; g < g1; ++g) {
                const int jb = g - g0;  // block-row within the tile
                uint32_t e = cur[g];
                while (e < p->row_ptr[g + 1] && p->col[e] < wend) {
                    // all stored blocks of this block-row in one aligned 4-column group
                    const int grp = (p->col[e] - wbeg) / 4;
                    uint32_t eg[4];
                    int n = 0;
                    while (e < p->row_ptr[g + 1] && p->col[e] < wend && (p->col[e] - wbeg) / 4 == grp)
                        eg[n++] = e++;
                    const int q = gq[grp], pt = gt[grp];
                    for (int sl = 0; sl < 2; ++sl) {
                        const int lo = 2 * sl, hi = std::min(n, lo + 2);
                        if (hi <= lo) continue;
                        used[sl] = true;
                        int pos[2];
                        uint32_t blk[2];
                        make_pair(p, eg + lo, hi - lo, pos, blk);
                        uint32_t &ix = idx[sl][jb * 4 + q];
                        ix &= ~(0xFu << (4 * pt));
                        ix |= (uint32_t)(pos[0] | (pos[1] << 2)) << (4 * pt);
                        for (int sp = 0; sp < 2; ++sp) {
                            if (blk[sp] == UINT32_MAX) continue;
                            for (int r = 0; r < 4; ++r)
                                op[sl][(16 * q + 4 * jb + r) * 16 + 2 * pt + sp] = p->vals[4 * (size_t)blk[sp] + r];
                        }
                    }
                }
                cur[g] = e;
            }
            memcpy(op[0] + 1024, idx[0], 64);
            memcpy(op[1] + 1024, idx[1], 64);
            memcpy(&ti.main[((size_t)w * ti.n_tiles + t) * kOpBytes], op[0], kOpBytes);
            if (used[0]) ti.n_entries++;
            if (used[1]) {
                ti.ovf.insert(ti.ovf.end(), op[1], op[1] + kOpBytes);
                ++n_ovf;
                ti.n_entries++;
                ti.n_overflow++;
            }
        }
        ti.ovf_ptr[(size_t)w * pstride + ti.n_tiles] = n_ovf;
    }
    return SL_OK;
}

sl_status build_host_image(const int8_t *w, int32_t n_out, int32_t k_in, const float *w_scale,
                           const float *bias, sl_packed_weight *p)
{
    try {
        p->n_out = n_out;
        p->k_in = k_in;
        p->w_scale.assign(w_scale, w_scale + n_out);
        if (bias)
            p->bias.assign(bias, bias + n_out);
        else
            p->bias.assign(n_out, 0.0f);
        sl_status st = build_bsr(w, n_out, k_in, p);
        if (st != SL_OK) return st;
        st = build_tiles(p);
        return st;
    } catch (const std::bad_alloc &) {
        set_error("host allocation failed while packing");
        return SL_ERR_OOM;
    }
}

// Inverse of build_tiles: every value of every operand is placed back at the
// (channel, column) the instruction reads it for. Fails on values beyond the
// matrix, two values at one position, or a pair whose two positions coincide.
static sl_status decode_operand(const int8_t *op, int32_t t, int32_t w, const sl_packed_weight *p, int8_t *dense)
{
    const int32_t k_in = p->k_in;
    for (int lane = 0; lane < 64; ++lane) {
        const int q = lane / 16, i = lane % 16, jb = i / 4;
        uint32_t ix;
        memcpy(&ix, op + 1024 + 4 * (jb * 4 + q), 4);
        for (int pt = 0; pt < 8; ++pt) {
            const int pos0 = (ix >> (4 * pt)) & 3, pos1 = (ix >> (4 * pt + 2)) & 3;
            for (int sp = 0; sp < 2; ++sp) {
                const int8_t v = op[lane * 16 + 2 * pt + sp];
                if (!v) continue;
                if (pos0 == pos1) {
                    set_error("tile image pair has two equal column positions");
                    return SL_ERR_INVALID_ARG;
                }
                const int32_t n = t * kTileN + i;
                const int32_t grp = w * (kWin / 4) + entry_group(q, pt);
                const int32_t col = 4 * grp + (sp ? pos1 : pos0);
                if (n >= p->n_out || col >= k_in) {
                    set_error("tile image holds a value outside the matrix");
                    return SL_ERR_INVALID_ARG;
                }
                int8_t &d = dense[(size_t)n * k_in + col];
                if (d) {
                    set_error("tile image places two values at one weight position");
                    return SL_ERR_INVALID_ARG;
                }
                d = v;
            }
        }
    }
    return SL_OK;
}

sl_status decode_tile_image(const sl_packed_weight *p, int8_t *dense)
{
    const TileImage &ti = p->tiles;
    const size_t pstride = (size_t)ti.n_tiles + 1;
    memset(dense, 0, (size_t)p->n_out * p->k_in);
    for (int32_t w = 0; w < ti.n_win; ++w) {
        for (int32_t t = 0; t < ti.n_tiles; ++t) {
            sl_status st = decode_operand(&ti.main[((size_t)w * ti.n_tiles + t) * kOpBytes], t, w, p, dense);
            if (st != SL_OK) return st;
            const uint32_t o0 = ti.ovf_ptr[(size_t)w * pstride + t], o1 = ti.ovf_ptr[(size_t)w * pstride + t + 1];
            if (o1 - o0 > 1) {
                set_error("tile image has more than one overflow operand for a (window, tile)");
                return SL_ERR_INVALID_ARG;
            }
            for (uint32_t o = o0; o < o1; ++o) {
                st = decode_operand(&ti.ovf[(size_t)o * kOpBytes], t, w, p, dense);
                if (st != SL_OK) return st;
            }
        }
    }
    return SL_OK;
}

}  // namespace sl
