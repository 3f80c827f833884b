// Internal definitions shared by the packer, the C-ABI layer and the kernels
// of the sparse INT8 linear library (gfx950). Not part of the public ABI.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/sparse_linear.h"

namespace sl {

// One channel tile = 16 output channels = 4 block-rows of 4x1 blocks. This is
// the row count of the 16x16x64 int8 matrix-core instruction's A operand.
constexpr int kTileN = 16;
// Contraction depth of one v_mfma_i32_16x16x64_i8: a tile's gathered column
// list is padded to a multiple of this.
constexpr int kStepK = 64;
// Input columns are processed in chunks of at most this many (one LDS stage).
constexpr int kChunkMax = 1024;
// Bytes of one k-step of the A-operand panel: 64 lanes x 16 int8.
constexpr int kStepBytes = 64 * 16;

struct TileImage {
    int32_t n_tiles = 0;
    int32_t kc = 0;        // chunk width (input columns per LDS stage)
    int32_t n_chunks = 0;  // ceil(k_in / kc)
    int64_t n_steps = 0;   // total k-steps over all (tile, chunk) segments
    int64_t union_cols = 0;
    int64_t padded_cols = 0;
    // segment (t, c) covers k-steps seg_ptr[t*n_chunks + c] .. seg_ptr[t*n_chunks + c + 1) - 1
    std::vector<uint32_t> seg_ptr;
    // A operand, per k-step: lane l holds 16 bytes; byte b of lane l is channel
    // 16t + (l % 16) at gathered position 16*(l/16) + b of the k-step.
    std::vector<int8_t> panel;
    // input column of each gathered position: [n_steps][64]
    std::vector<uint16_t> ucol;
};

struct DeviceImage {
    int device = -1;
    void *base = nullptr;  // one allocation holding everything below
    const uint32_t *seg_ptr = nullptr;
    const int8_t *panel = nullptr;
    const uint16_t *ucol = nullptr;
    const float *w_scale = nullptr;
    const float *bias = nullptr;
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

// thread-local error text
void set_error(const std::string &msg);
void clear_error();

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
sl_status launch_linear(const sl_packed_weight *w, const int8_t *x, int64_t m, float sx, int32_t kind,
                        float inv_so, void *y, void *stream);
sl_status launch_quantize(const float *x, int64_t n, float inv_scale, int8_t *q, void *stream);

}  // namespace sl
