// Internal definitions shared by the packer, the C-ABI layer and the kernels
// of the sparse INT8 linear library (gfx950). Not part of the public ABI.
#pragma once

#include <stdint.h>

#include <memory>
#include <string>
#include <vector>

#include "../../include/sparse_linear.h"

namespace sl {

// One channel tile = 16 output channels = 4 block-rows of 4x1 blocks: the
// row count of the 4:2-sparse int8 matrix-core instruction
// v_smfmac_i32_16x16x128_i8 (A: 16 rows x 128 columns with at most 2 stored
// values in every aligned group of 4 columns; B: 128 x 16 dense).
constexpr int kTileN = 16;
// Input columns per window (the contraction depth of one instruction).
constexpr int kWin = 128;
// Column group (of 4 consecutive window columns) that value pair t of a lane
// in lane group q (q = lane / 16) addresses, as the instruction defines it:
// the B operand's lane group g holds window columns 32g .. 32g+31 of its token.
inline int entry_group(int q, int t) { return 8 * (2 * (q & 1) + (t >> 2)) + 4 * (q >> 1) + (t & 3); }

// One instruction operand in the image: 64 lanes x 16 value bytes (lane
// 16q + i holds row i; byte 2p + s is slot s of value pair p, addressing
// window column 4 * entry_group(q, p) + its 2-bit index), then the index words
// of the 16 (block-row jb, lane group q) pairs at word 4 * jb + q (the 4 rows
// of a block-row share their column positions).
constexpr int kOpBytes = 64 * 16 + 16 * 4;  // 1088 = 68 pieces of 16 bytes
constexpr int kOpPieces = kOpBytes / 16;

// GPU image of a packed weight. Per (128-column window w, 16-channel tile t)
// the main operand holds the first two stored blocks of every (block-row,
// aligned 4-column group); where a group holds 3 or 4, an overflow operand on
// the same window holds the rest.
//   main     [n_win][n_tiles] operands (all-zero where a tile stores nothing)
//   ovf      overflow operands, window-major then tile
//   ovf_ptr  [n_win][n_tiles + 1]: overflow operands of (w, t) are
//            ovf_ptr[w][t] .. ovf_ptr[w][t+1]-1 (0 or 1 of them)
struct TileImage {
    int32_t n_tiles = 0;
    int32_t n_win = 0;       // ceil(k_in / 128)
    int64_t n_entries = 0;   // operands holding a stored block = instructions per 16 tokens
    int64_t n_overflow = 0;  // overflow operands
    std::vector<int8_t> main;
    std::vector<int8_t> ovf;
    std::vector<uint32_t> ovf_ptr;
};


// Step table of the fused GELU(erf) + int8 requantisation (gelu_table.cpp).
constexpr int kGeluCells = 448;
struct alignas(8) GeluCell {
    float thr;     // first y of the cell whose code is q_hi (+inf: none)
    int8_t q_lo;   // code of the cell's y below thr
    int8_t q_hi;   // code from thr on
    int16_t pad;
};
// The cell of y is read off the bits of one fused multiply-add: off carries
// kGeluBase = 2^23, where consecutive fp32 values are consecutive integers, so
// t = med3(fma(y, hinv, off), kGeluBase, kGeluBase + nc - 1) is kGeluBase
// plus the cell index (the fma rounds to nearest even), and the index is
// bits(t) - bits(kGeluBase), which is also the low 24 bits of bits(t): no
// float-to-int conversion.
constexpr float kGeluBase = 8388608.0f;
struct GeluTable {
    float hinv = 0, off = 0;  // cell(y) = med3(fma(y, hinv, off), kGeluBase, kGeluBase + nc - 1) - kGeluBase
    int32_t nc = 0;
    bool ok = false;          // false: a cell would hold two changes; use erf
    GeluCell cell[kGeluCells];
};
// The step table for inverse output scale inv_so from a fixed-size cache
// (built on first use of inv_so, under a lock; no allocation), copied into
// *out. Returns out->ok.
bool gelu_table(float inv_so, GeluTable *out);
// the code the table gives for y (host copy of the kernels' lookup)
int gelu_table_code(const GeluTable &t, float y);

// Per tile-group size nt (channel tiles per workgroup): for every window w and
// group g, the pair (mask, first): bit j of mask set if tile g*nt + j has an
// overflow operand in window w; first = index of the group's first overflow
// operand of the window. Layout [n_win][n_groups][2] uint32.
constexpr int kMaxOmTables = 8;

// Weight panels of the weight-stationary kernel, per tile-group size nt: for
// channel group g and window w, the entry {mask, first, base, 0} at
// [g][n_win + 1][4] uint32: mask and first as in the overflow table; base =
// offset, in 16-byte pieces, of the window's operands in the group's panel
// (the nt main operands, then nt overflow operand slots, one per tile, zeros
// where the tile has none: base = w * 2 * nt * 68). Entry n_win holds the
// panel's total size in its base word.
constexpr int kMaxPanTables = 4;

struct DeviceImage {
    int device = -1;
    void *base = nullptr;  // one allocation holding everything below
    const int8_t *main = nullptr;
    const int8_t *ovf = nullptr;
    const uint32_t *ovf_ptr = nullptr;
    const float *w_scale = nullptr;
    const float *bias = nullptr;
    int32_t n_om = 0;
    int32_t om_nt[kMaxOmTables] = {};
    const uint32_t *om[kMaxOmTables] = {};
    int32_t n_pan = 0;
    int32_t pan_nt[kMaxPanTables] = {};
    int32_t pan_pieces[kMaxPanTables] = {};  // largest panel over the groups, 16-byte pieces
    // per channel-group size: each group's window table ([n_win + 1][4]
    // words: overflow mask, first overflow operand, panel offset in pieces)
    // followed by its panel, byte for byte as the weight-stationary kernel
    // holds them in LDS, groups pan_stride bytes apart (a multiple of 1024;
    // 0: the panels do not fit in LDS and there is no such image)
    uint32_t pan_stride[kMaxPanTables] = {};
    const int8_t *pan[kMaxPanTables] = {};
    // split-reduction kernel: the overflow operands in the main image's
    // order, one slot per (window, tile), zeros where the tile has none
    const int8_t *ovfd = nullptr;
    uint32_t ovfd_bytes = 0;
    int64_t bytes = 0;
};

}  // namespace sl

struct sl_packed_weight {
    int32_t n_out = 0;
    int32_t k_in = 0;
    int64_t nnzb = 0;
    // canonical BSR, 4x1 blocks
    std::vector<uint32_t> row_ptr;
    std::vector<uint16_t> col;
    std::vector<int8_t> vals;
    std::vector<float> w_scale;
    std::vector<float> bias;  // zeros when the caller passed NULL
    sl::TileImage tiles;
    bool on_device = false;
    sl::DeviceImage dev;
};

namespace sl {

// thread-local name of the last launched kernel shape (sl_last_path), written
// printf-style into a fixed buffer: no allocation on the run path
void set_last_path(const char *fmt, ...) __attribute__((format(printf, 1, 2)));
void append_last_path(const char *text);
const char *last_path();

// thread-local error text, printf-style into a fixed buffer
void set_error(const char *fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

// Kernel-choice overrides for tests and tuning (SL_PATH, SL_TILE, SL_DTILE,
// SL_PTILE), read from the environment once and again on sl_reload_env()
struct EnvCfg {
    char path[16];  // "" (automatic), "split", "panel", "direct", "staged"
    int tile[5];    // SL_TILE "st,ct,wm,wn,d"; tile[0] == 0: unset
    int dtile[4];   // SL_DTILE "st,nt,wm,d"
    int ptile[4];   // SL_PTILE "nt,st,nwv,r"
    int pslices;    // SL_PSLICES: token slices of the weight-stationary kernel (0: its cost model picks)
};
const EnvCfg &env_cfg();
void reload_env();

// host packer (pack.cpp)
sl_status validate_weight_args(const int8_t *w, int32_t n_out, int32_t k_in, int32_t bh, int32_t bw,
                               const float *w_scale, const float *bias);
sl_status build_host_image(const int8_t *w, int32_t n_out, int32_t k_in, const float *w_scale,
                           const float *bias, sl_packed_weight *out);
sl_status decode_tile_image(const sl_packed_weight *w, int8_t *dense);

// device side (kernels.hip)
sl_status upload_image(sl_packed_weight *w);
void release_image(sl_packed_weight *w);
sl_status check_device_arch(int *device);
sl_status launch_linear(const sl_packed_weight *w, const int8_t *x, int32_t x_layout, int64_t m, float sx,
                        int32_t kind, float inv_so, void *y, int32_t y_layout, void *stream);
sl_status launch_quantize(const float *x, int64_t n, float inv_scale, int8_t *q, void *stream);
sl_status launch_quantize_t16x32(const float *x, int64_t rows, int32_t cols, float inv_scale, int8_t *q,
                                 void *stream);

}  // namespace sl
