// Host packer: dense int8 weight -> canonical 4x1 BSR -> GPU tile image.
//
// Section "Sparse GEMM operators": the sparse weight is stored compressed and
// its mask (the column index of every stored block) drives the
// reorganisation of the input. Appendix "Block-wise structured sparsity": the
// blocks are 1-D, 4 consecutive output rows at one input column.
//
// The GPU image regroups 4 block-rows into a 16-channel tile so that one
// 16x16x64 int8 matrix-core instruction can take them as its A operand: per
// (tile, k-chunk) the union of the 4 block-rows' stored columns is listed once,
// padded to a multiple of 64, and the 16 x |union| weight panel is laid out in
// the order the instruction's lanes read it (16 bytes per lane per k-step).
// Positions a block-row does not store hold 0, so the int32 sum is unchanged.
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
            set_error("w_scale must be finite and > 0 (channel " + std::to_string(n) + ")");
            return SL_ERR_INVALID_ARG;
        }
        if (bias && !isfinite(bias[n])) {
            set_error("bias must be finite (channel " + std::to_string(n) + ")");
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

static sl_status build_tiles(sl_packed_weight *p)
{
    TileImage &ti = p->tiles;
    const int32_t nbr = p->n_out / 4;
    const int32_t k_in = p->k_in;
    ti.n_tiles = (p->n_out + kTileN - 1) / kTileN;
    ti.kc = std::min<int32_t>(k_in, kChunkMax);
    ti.n_chunks = (k_in + ti.kc - 1) / ti.kc;
    ti.seg_ptr.assign((size_t)ti.n_tiles * ti.n_chunks + 1, 0);
    ti.panel.clear();
    ti.ucol.clear();
    ti.union_cols = 0;
    ti.padded_cols = 0;

    std::vector<uint16_t> uni;
    std::vector<int32_t> where(k_in, -1);  // position of a column in the current union
    uint32_t step = 0;
    for (int32_t t = 0; t < ti.n_tiles; ++t) {
        const int32_t g0 = 4 * t, g1 = std::min(4 * t + 4, nbr);
        // cursors into each block-row's ascending column list
        uint32_t cur[4] = {0, 0, 0, 0};
        for (int32_t g = g0; g < g1; ++g) cur[g - g0] = p->row_ptr[g];
        for (int32_t c = 0; c < ti.n_chunks; ++c) {
            const int32_t kbeg = c * ti.kc, kend = std::min(k_in, kbeg + ti.kc);
            uni.clear();
            uint32_t stop[4];
            for (int32_t g = g0; g < g1; ++g) {
                uint32_t e = cur[g - g0];
                while (e < p->row_ptr[g + 1] && p->col[e] < kend) {
                    uni.push_back(p->col[e]);
                    ++e;
                }
                stop[g - g0] = e;
            }
            std::sort(uni.begin(), uni.end());
            uni.erase(std::unique(uni.begin(), uni.end()), uni.end());
            const int64_t nu = (int64_t)uni.size();
            const int64_t nsteps = (nu + kStepK - 1) / kStepK;
            ti.union_cols += nu;
            ti.padded_cols += nsteps * kStepK;
            for (int64_t i = 0; i < nu; ++i) where[uni[i]] = (int32_t)i;
            // column list, padded with the chunk's first column (weight 0 there)
            const size_t ubase = ti.ucol.size();
            ti.ucol.resize(ubase + nsteps * kStepK, (uint16_t)kbeg);
            for (int64_t i = 0; i < nu; ++i) ti.ucol[ubase + i] = uni[i];
            // panel: position i of the segment lives in k-step i/64, at
            // lane group (i%64)/16, byte (i%16); row r of the tile = lane%16
            const size_t pbase = ti.panel.size();
            ti.panel.resize(pbase + nsteps * kStepBytes, 0);
            for (int32_t g = g0; g < g1; ++g) {
                for (uint32_t e = cur[g - g0]; e < stop[g - g0]; ++e) {
                    const int64_t pos = where[p->col[e]];
                    const int64_t s = pos / kStepK, q = pos % kStepK;
                    const int64_t grp = q / 16, byte = q % 16;
                    for (int r = 0; r < 4; ++r) {
                        const int64_t row = 4 * (g - g0) + r;  // 0..15 within the tile
                        const int64_t lane = grp * 16 + row;
                        ti.panel[pbase + s * kStepBytes + lane * 16 + byte] = p->vals[4 * e + r];
                    }
                }
                cur[g - g0] = stop[g - g0];
            }
            for (int64_t i = 0; i < nu; ++i) where[uni[i]] = -1;
            step += (uint32_t)nsteps;
            ti.seg_ptr[(size_t)t * ti.n_chunks + c + 1] = step;
        }
    }
    ti.n_steps = step;
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
        return build_tiles(p);
    } catch (const std::bad_alloc &) {
        set_error("host allocation failed while packing");
        return SL_ERR_OOM;
    }
}

// Inverse of build_tiles: place every panel byte back at (channel, column).
// Fails if a (channel, column) pair would receive two non-zero values.
sl_status decode_tile_image(const sl_packed_weight *p, int8_t *dense)
{
    const TileImage &ti = p->tiles;
    const int32_t k_in = p->k_in;
    memset(dense, 0, (size_t)p->n_out * k_in);
    for (int32_t t = 0; t < ti.n_tiles; ++t) {
        for (int32_t c = 0; c < ti.n_chunks; ++c) {
            const uint32_t s0 = ti.seg_ptr[(size_t)t * ti.n_chunks + c];
            const uint32_t s1 = ti.seg_ptr[(size_t)t * ti.n_chunks + c + 1];
            for (uint32_t s = s0; s < s1; ++s) {
                for (int lane = 0; lane < 64; ++lane) {
                    const int row = lane % 16, grp = lane / 16;
                    const int32_t n = t * kTileN + row;
                    for (int b = 0; b < 16; ++b) {
                        const int8_t v = ti.panel[(size_t)s * kStepBytes + lane * 16 + b];
                        if (!v) continue;
                        if (n >= p->n_out) {
                            set_error("tile image holds a value beyond n_out");
                            return SL_ERR_INVALID_ARG;
                        }
                        const int32_t u = ti.ucol[(size_t)s * kStepK + grp * 16 + b];
                        if (u < c * ti.kc || u >= std::min(k_in, (c + 1) * ti.kc)) {
                            set_error("tile image column outside its chunk");
                            return SL_ERR_INVALID_ARG;
                        }
                        int8_t &d = dense[(size_t)n * k_in + u];
                        if (d) {
                            set_error("tile image places two values at one weight position");
                            return SL_ERR_INVALID_ARG;
                        }
                        d = v;
                    }
                }
            }
        }
    }
    return SL_OK;
}

}  // namespace sl
