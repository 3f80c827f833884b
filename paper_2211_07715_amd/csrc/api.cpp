// C-ABI layer of the sparse INT8 linear library: argument checks, handle
// lifetime and dispatch to the gfx950 kernels. No exception crosses the ABI.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <new>

#include "sl_internal.h"

namespace sl {

static thread_local char g_last_error[512];
static thread_local char g_last_path[192];

void set_error(const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
}
void clear_error() { g_last_error[0] = 0; }

void set_last_path(const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_path, sizeof(g_last_path), fmt, ap);
    va_end(ap);
}
void append_last_path(const char *text)
{
    const size_t n = strlen(g_last_path);
    snprintf(g_last_path + n, sizeof(g_last_path) - n, "%s", text);
}
const char *last_path() { return g_last_path; }

static EnvCfg g_env;
static std::once_flag g_env_once;

static void parse_ints(const char *v, int *out, int n)
{
    int tmp[5] = {};
    const int got = v ? sscanf(v, "%d,%d,%d,%d,%d", &tmp[0], &tmp[1], &tmp[2], &tmp[3], &tmp[4]) : 0;
    for (int i = 0; i < n; ++i) out[i] = got >= n ? tmp[i] : 0;
}

void reload_env()
{
    EnvCfg e{};
    const char *p = getenv("SL_PATH");
    if (p) snprintf(e.path, sizeof(e.path), "%s", p);
    parse_ints(getenv("SL_TILE"), e.tile, 5);
    parse_ints(getenv("SL_DTILE"), e.dtile, 4);
    parse_ints(getenv("SL_PTILE"), e.ptile, 4);
    parse_ints(getenv("SL_PSLICES"), &e.pslices, 1);
    g_env = e;
}

const EnvCfg &env_cfg()
{
    std::call_once(g_env_once, reload_env);
    return g_env;
}

}  // namespace sl

using namespace sl;

// Runs one entry point's body; an exception (a failed host allocation, a
// failed lock) becomes a status and a message instead of crossing the ABI.
template <class F>
static sl_status guarded(F &&body)
{
    try {
        return body();
    } catch (const std::bad_alloc &) {
        set_error("host allocation failed");
        return SL_ERR_OOM;
    } catch (const std::exception &ex) {
        set_error("internal error: %s", ex.what());
        return SL_ERR_HIP;
    } catch (...) {
        set_error("internal error");
        return SL_ERR_HIP;
    }
}

static sl_status pack_common(const int8_t *w_host, int32_t n_out, int32_t k_in, int32_t block_h,
                             int32_t block_w, const float *w_scale_host, const float *bias_host,
                             sl_packed_weight **out, bool upload)
{
    clear_error();
    if (!out) {
        set_error("out must not be NULL");
        return SL_ERR_INVALID_ARG;
    }
    *out = nullptr;
    sl_status st = validate_weight_args(w_host, n_out, k_in, block_h, block_w, w_scale_host, bias_host);
    if (st != SL_OK) return st;
    int device = -1;
    if (upload) {
        st = check_device_arch(&device);
        if (st != SL_OK) return st;
    }
    // freed on every way out but success, an exception included
    struct Holder {
        sl_packed_weight *p;
        ~Holder() { sparse_linear_free(p); }
    } h{new (std::nothrow) sl_packed_weight()};
    if (!h.p) {
        set_error("host allocation failed");
        return SL_ERR_OOM;
    }
    st = build_host_image(w_host, n_out, k_in, w_scale_host, bias_host, h.p);
    if (st == SL_OK && upload) {
        h.p->dev.device = device;
        st = upload_image(h.p);
    }
    if (st != SL_OK) return st;
    *out = h.p;
    h.p = nullptr;
    return SL_OK;
}

extern "C" {

sl_status sparse_linear_pack(const int8_t *w_host, int32_t n_out, int32_t k_in, int32_t block_h,
                             int32_t block_w, const float *w_scale_host, const float *bias_host,
                             sl_packed_weight **out)
{
    return guarded([&] { return pack_common(w_host, n_out, k_in, block_h, block_w, w_scale_host, bias_host, out, true); });
}

sl_status sparse_linear_pack_host(const int8_t *w_host, int32_t n_out, int32_t k_in, int32_t block_h,
                                  int32_t block_w, const float *w_scale_host, const float *bias_host,
                                  sl_packed_weight **out)
{
    return guarded([&] { return pack_common(w_host, n_out, k_in, block_h, block_w, w_scale_host, bias_host, out, false); });
}

static bool good_scale(float s) { return isfinite(s) && s > 0.0f; }

static sl_status run_layout_impl(const sl_packed_weight *w, const int8_t *x_dev, int32_t x_layout,
                                 int64_t m_tokens, float x_scale, int32_t epilogue_kind, float out_scale,
                                 void *y_dev, int32_t y_layout, void *hip_stream)
{
    clear_error();
    if (!w) {
        set_error("w must not be NULL");
        return SL_ERR_INVALID_ARG;
    }
    if (!w->on_device) {
        set_error("handle was packed with sparse_linear_pack_host; pack it on a device to run");
        return SL_ERR_NOT_ON_DEVICE;
    }
    if (epilogue_kind < SL_EPI_ACC_I32 || epilogue_kind > SL_EPI_I8_GELU) {
        set_error("unknown epilogue kind %d", epilogue_kind);
        return SL_ERR_INVALID_ARG;
    }
    if (x_layout != SL_LAYOUT_ROWS && x_layout != SL_LAYOUT_T16X32) {
        set_error("unknown x_layout %d", x_layout);
        return SL_ERR_INVALID_ARG;
    }
    if (y_layout != SL_LAYOUT_ROWS && y_layout != SL_LAYOUT_T16X32) {
        set_error("unknown y_layout %d", y_layout);
        return SL_ERR_INVALID_ARG;
    }
    if (m_tokens < 0) {
        set_error("m_tokens must be >= 0");
        return SL_ERR_SHAPE;
    }
    if (epilogue_kind != SL_EPI_ACC_I32 && !good_scale(x_scale)) {
        set_error("x_scale must be finite and > 0");
        return SL_ERR_INVALID_ARG;
    }
    const bool i8 = epilogue_kind == SL_EPI_I8 || epilogue_kind == SL_EPI_I8_GELU;
    if (i8 && !good_scale(out_scale)) {
        set_error("out_scale must be finite and > 0 for the int8 epilogues");
        return SL_ERR_INVALID_ARG;
    }
    if (y_layout == SL_LAYOUT_T16X32 && !i8) {
        set_error("y_layout SL_LAYOUT_T16X32 is for the int8 epilogues only");
        return SL_ERR_INVALID_ARG;
    }
    if (m_tokens == 0) return SL_OK;
    if (!x_dev || !y_dev) {
        set_error("x_dev and y_dev must not be NULL");
        return SL_ERR_INVALID_ARG;
    }
    if (x_layout == SL_LAYOUT_T16X32 && reinterpret_cast<uintptr_t>(x_dev) % 16) {
        set_error("x_dev must be 16-byte aligned for SL_LAYOUT_T16X32");
        return SL_ERR_INVALID_ARG;
    }
    const uintptr_t need = (i8 && y_layout == SL_LAYOUT_ROWS) ? 4 : 16;
    if (reinterpret_cast<uintptr_t>(y_dev) % need) {
        set_error("y_dev must be %d-byte aligned for this epilogue and layout", (int)need);
        return SL_ERR_INVALID_ARG;
    }
    // fl(1/so), one fp32 division, as the definition states
    const float inv_so = i8 ? 1.0f / out_scale : 1.0f;
    return launch_linear(w, x_dev, x_layout, m_tokens, x_scale, epilogue_kind, inv_so, y_dev, y_layout,
                         hip_stream);
}

sl_status sparse_linear_run_layout(const sl_packed_weight *w, const int8_t *x_dev, int32_t x_layout,
                                   int64_t m_tokens, float x_scale, int32_t epilogue_kind, float out_scale,
                                   void *y_dev, int32_t y_layout, void *hip_stream)
{
    return guarded([&] {
        return run_layout_impl(w, x_dev, x_layout, m_tokens, x_scale, epilogue_kind, out_scale, y_dev, y_layout,
                               hip_stream);
    });
}

sl_status sparse_linear_run(const sl_packed_weight *w, const int8_t *x_dev, int64_t m_tokens,
                            float x_scale, int32_t epilogue_kind, float out_scale, void *y_dev,
                            void *hip_stream)
{
    return sparse_linear_run_layout(w, x_dev, SL_LAYOUT_ROWS, m_tokens, x_scale, epilogue_kind, out_scale, y_dev,
                                    SL_LAYOUT_ROWS, hip_stream);
}

sl_status quantize_act(const float *x_dev, int64_t numel, float scale, int8_t *q_dev, void *hip_stream)
{
    clear_error();
    if (numel < 0) {
        set_error("numel must be >= 0");
        return SL_ERR_SHAPE;
    }
    if (!good_scale(scale)) {
        set_error("scale must be finite and > 0");
        return SL_ERR_INVALID_ARG;
    }
    if (numel == 0) return SL_OK;
    if (!x_dev || !q_dev) {
        set_error("x_dev and q_dev must not be NULL");
        return SL_ERR_INVALID_ARG;
    }
    const float inv = 1.0f / scale;
    return launch_quantize(x_dev, numel, inv, q_dev, hip_stream);
}

sl_status quantize_act_layout(const float *x_dev, int64_t rows, int32_t cols, float scale, int8_t *q_dev,
                              int32_t q_layout, void *hip_stream)
{
    clear_error();
    if (rows < 0 || cols < 0) {
        set_error("rows and cols must be >= 0");
        return SL_ERR_SHAPE;
    }
    if (q_layout != SL_LAYOUT_ROWS && q_layout != SL_LAYOUT_T16X32) {
        set_error("unknown q_layout %d", q_layout);
        return SL_ERR_INVALID_ARG;
    }
    if (q_layout == SL_LAYOUT_ROWS) return quantize_act(x_dev, rows * (int64_t)cols, scale, q_dev, hip_stream);
    if (!good_scale(scale)) {
        set_error("scale must be finite and > 0");
        return SL_ERR_INVALID_ARG;
    }
    if (rows == 0 || cols == 0) return SL_OK;
    if (!x_dev || !q_dev) {
        set_error("x_dev and q_dev must not be NULL");
        return SL_ERR_INVALID_ARG;
    }
    if (reinterpret_cast<uintptr_t>(q_dev) % 16 || reinterpret_cast<uintptr_t>(x_dev) % 4) {
        set_error("q_dev must be 16-byte and x_dev 4-byte aligned for SL_LAYOUT_T16X32");
        return SL_ERR_INVALID_ARG;
    }
    const float inv = 1.0f / scale;
    return launch_quantize_t16x32(x_dev, rows, cols, inv, q_dev, hip_stream);
}

sl_status sparse_linear_unpack(const sl_packed_weight *w, int8_t *w_host)
{
    clear_error();
    if (!w || !w_host) {
        set_error("w and w_host must not be NULL");
        return SL_ERR_INVALID_ARG;
    }
    return guarded([&] { return decode_tile_image(w, w_host); });
}

sl_status sparse_linear_info(const sl_packed_weight *w, int32_t *n_out, int32_t *k_in, int64_t *nnz_blocks)
{
    clear_error();
    if (!w) {
        set_error("w must not be NULL");
        return SL_ERR_INVALID_ARG;
    }
    if (n_out) *n_out = w->n_out;
    if (k_in) *k_in = w->k_in;
    if (nnz_blocks) *nnz_blocks = w->nnzb;
    return SL_OK;
}

sl_status sparse_linear_export_bsr(const sl_packed_weight *w, uint32_t *row_ptr, uint16_t *col, int8_t *vals)
{
    clear_error();
    if (!w) {
        set_error("w must not be NULL");
        return SL_ERR_INVALID_ARG;
    }
    if (row_ptr) memcpy(row_ptr, w->row_ptr.data(), w->row_ptr.size() * sizeof(uint32_t));
    if (col && !w->col.empty()) memcpy(col, w->col.data(), w->col.size() * sizeof(uint16_t));
    if (vals && !w->vals.empty()) memcpy(vals, w->vals.data(), w->vals.size());
    return SL_OK;
}

sl_status sparse_linear_tile_stats(const sl_packed_weight *w, int32_t *n_tiles, int64_t *n_entries,
                                   int64_t *n_overflow, int64_t *image_bytes)
{
    clear_error();
    if (!w) {
        set_error("w must not be NULL");
        return SL_ERR_INVALID_ARG;
    }
    const TileImage &ti = w->tiles;
    if (n_tiles) *n_tiles = ti.n_tiles;
    if (n_entries) *n_entries = ti.n_entries;
    if (n_overflow) *n_overflow = ti.n_overflow;
    if (image_bytes)
        *image_bytes = (int64_t)(ti.main.size() + ti.ovf.size() + ti.ovf_ptr.size() * 4 + (size_t)w->n_out * 8);
    return SL_OK;
}

void sparse_linear_free(sl_packed_weight *w)
{
    if (!w) return;
    if (w->on_device) release_image(w);
    delete w;
}

const char *sl_status_string(int32_t s)
{
    switch (s) {
    case SL_OK: return "SL_OK";
    case SL_ERR_INVALID_ARG: return "SL_ERR_INVALID_ARG";
    case SL_ERR_SHAPE: return "SL_ERR_SHAPE";
    case SL_ERR_HIP: return "SL_ERR_HIP";
    case SL_ERR_OOM: return "SL_ERR_OOM";
    case SL_ERR_UNSUPPORTED: return "SL_ERR_UNSUPPORTED";
    case SL_ERR_NOT_ON_DEVICE: return "SL_ERR_NOT_ON_DEVICE";
    default: return "SL_ERR_UNKNOWN";
    }
}

const char *sl_last_error(void) { return g_last_error; }

int32_t sl_abi_version(void) { return SL_ABI_VERSION; }

const char *sl_last_path(void) { return sl::last_path(); }

void sl_reload_env(void)
{
    try {
        sl::env_cfg();  // (the first read, if not yet done)
        sl::reload_env();
    } catch (...) {
    }
}

sl_status sl_gelu_table_codes(float out_scale, const float *y, int8_t *q, int64_t n)
{
    clear_error();
    if (!good_scale(out_scale)) {
        set_error("out_scale must be finite and > 0");
        return SL_ERR_INVALID_ARG;
    }
    if (n < 0 || (n > 0 && (!y || !q))) {
        set_error("y and q must not be NULL, n >= 0");
        return SL_ERR_INVALID_ARG;
    }
    return guarded([&] {
        GeluTable t;
        if (!gelu_table(1.0f / out_scale, &t)) {
            set_error("no step table for this out_scale; the kernels evaluate erf");
            return SL_ERR_UNSUPPORTED;
        }
        for (int64_t i = 0; i < n; ++i) q[i] = (int8_t)gelu_table_code(t, y[i]);
        return SL_OK;
    });
}

}  // extern "C"
