/*
 * sparse_linear.h -- C ABI of the MI355X (gfx950) sparse INT8 linear layer.
 *
 * The operation is the one the paper accelerates with its INT8 sparse GEMM
 * (Section "Sparse GEMM operators", Figure 1, Algorithm 1): a dense, quantised
 * int8 input multiplied by an int8 weight that is block-sparse in 1-D blocks
 * of 4 consecutive output rows (Appendix "Block-wise structured sparsity"),
 * accumulated in int32, followed by fused post-operators (bias, GELU,
 * downconvert; Appendix "Graph optimization" and Algorithm 1's
 * "downconvert and post-operator fusion").
 *
 * Shapes and layouts (row-major and contiguous unless a call takes an
 * sl_layout, below):
 *   X  [m_tokens x k_in]   int8, device memory     (tokens x input features)
 *   W  [n_out    x k_in]   int8, host memory       (output x input features)
 *   Y  [m_tokens x n_out]  int32 | fp32 | int8, device memory, per epilogue
 *
 * Per output element, with acc = sum_k X[m][k] * W[n][k] (exact int32):
 *   SL_EPI_ACC_I32 : Y = acc
 *   SL_EPI_F32     : Y = (float)acc * (x_scale * w_scale[n]) + bias[n]
 *   SL_EPI_F32_GELU: Y = GELU_erf(above)
 *   SL_EPI_I8      : Y = clamp(rint(above_f32 * (1 / out_scale)), -127, 127)
 *   SL_EPI_I8_GELU : Y = clamp(rint(GELU_erf(...) * (1 / out_scale)), -127, 127)
 * (fp32 arithmetic; GELU_erf(y) = 0.5 * y * (1 + erf(y / sqrt 2)); rint rounds
 * half to even; symmetric int8, zero point 0, never -128.)
 *
 * Errors: every function returns an sl_status; nothing aborts and no C++
 * exception crosses this boundary. sl_last_error() gives a thread-local text
 * for the last failure on the calling thread.
 */
#ifndef SPARSE_LINEAR_H
#define SPARSE_LINEAR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SL_ABI_VERSION 3

typedef enum {
    SL_OK = 0,
    SL_ERR_INVALID_ARG = -1, /* NULL pointer, unknown kind, bad scale, block shape != 4x1 */
    SL_ERR_SHAPE = -2,       /* n_out % 4 != 0, k_in outside [1, 65535], m_tokens < 0    */
    SL_ERR_HIP = -3,         /* a HIP runtime call failed; text in sl_last_error()     */
    SL_ERR_OOM = -4,         /* host or device allocation failed                        */
    SL_ERR_UNSUPPORTED = -5, /* device is not gfx950, or a size this build cannot run   */
    SL_ERR_NOT_ON_DEVICE = -6 /* handle from sparse_linear_pack_host used with run      */
} sl_status;

typedef enum {
    SL_EPI_ACC_I32 = 0, /* raw int32 accumulators                              */
    SL_EPI_F32 = 1,     /* dequant + bias -> fp32                              */
    SL_EPI_F32_GELU = 2,/* dequant + bias + GELU(erf) -> fp32                  */
    SL_EPI_I8 = 3,      /* dequant + bias -> requantised int8                   */
    SL_EPI_I8_GELU = 4  /* dequant + bias + GELU(erf) -> requantised int8       */
} sl_epilogue_kind;

/*
 * Layouts of an int8 activation tensor of `rows` tokens x `cols` features
 * (the input X of a layer, or the int8 output Y that feeds the next layer):
 *   SL_LAYOUT_ROWS    row-major: element (t, c) at byte t * cols + c.
 *   SL_LAYOUT_T16X32  blocks of 16 tokens x 32 features, each block 512
 *                     contiguous bytes, token-major inside: element (t, c) at
 *                     byte ((t / 16) * C + c / 32) * 512 + (t % 16) * 32 + c % 32
 *                     with C = ceil(cols / 32); the tensor occupies
 *                     ceil(rows / 16) * C * 512 bytes. Bytes of padding
 *                     tokens (t >= rows) and padding features (c >= cols)
 *                     may hold anything: a layer never lets them reach a
 *                     stored output (padding features meet zero weights).
 * T16X32 is the order in which the matrix cores consume the dense operand
 * (16 tokens per instruction, 32 consecutive features per lane), so a layer
 * reads it with whole cache lines per group of lanes; a chain of layers can
 * keep its activations in it from the first quantisation to the last
 * int8 output.
 */
typedef enum {
    SL_LAYOUT_ROWS = 0,
    SL_LAYOUT_T16X32 = 1
} sl_layout;

/* Opaque packed weight. Immutable after packing: any number of threads and
 * streams may run with one handle at once (the paper's weight sharing across
 * parallel inference instances, Section "Advanced runtime" and Appendix
 * "Weight sharing"). */
typedef struct sl_packed_weight sl_packed_weight;

/*
 * Pack a dense block-sparse int8 weight for the current HIP device.
 * Section "Sparse GEMM operators": non-zero weight blocks are stored
 * compressed, with the mask (column indices) that drives the input gather.
 *   w_host        [n_out x k_in] int8, row-major; a 4x1 block (rows 4g..4g+3,
 *                 column k) is stored iff one of its 4 values is non-zero.
 *   n_out         multiple of 4 (Algorithm 1's padding remark: sizes not
 *                 divisible by 4 are not handled) -> else SL_ERR_SHAPE.
 *   k_in          1 .. 65535 -> else SL_ERR_SHAPE.
 *   block_h, block_w  must be 4 and 1 -> else SL_ERR_INVALID_ARG.
 *   w_scale_host  [n_out] per-output-channel fp32 scale, finite and > 0.
 *   bias_host     [n_out] fp32, or NULL for zero bias.
 *   out           receives the handle; *out is set to NULL on failure.
 * Copies everything it needs (the caller keeps ownership of its buffers),
 * allocates device memory with hipMalloc and synchronises the upload.
 * Returns SL_ERR_UNSUPPORTED when the current device is not gfx950.
 */
sl_status sparse_linear_pack(const int8_t *w_host, int32_t n_out, int32_t k_in, int32_t block_h,
                             int32_t block_w, const float *w_scale_host, const float *bias_host,
                             sl_packed_weight **out);

/*
 * Same validation and packing as sparse_linear_pack, host memory only: no HIP
 * call is made, so it works without a GPU. The handle supports
 * sparse_linear_info / _unpack / _export_bsr / _tile_stats / _free;
 * sparse_linear_run on it returns SL_ERR_NOT_ON_DEVICE.
 */
sl_status sparse_linear_pack_host(const int8_t *w_host, int32_t n_out, int32_t k_in, int32_t block_h,
                                  int32_t block_w, const float *w_scale_host, const float *bias_host,
                                  sl_packed_weight **out);

/*
 * Y = epilogue(X * W^T) on hip_stream (asynchronous; never synchronises,
 * allocates nothing). The hot path: Section "Sparse GEMM operators" -- the
 * input columns selected by the weight's mask are gathered, multiplied with
 * the stored blocks in int8 with int32 accumulation, and bias and the other
 * post-operators are applied before the single store of Y.
 *   w             handle from sparse_linear_pack, packed on the current device.
 *   x_dev         [m_tokens x k_in] int8 device pointer.
 *   m_tokens      >= 0; 0 is a no-op returning SL_OK.
 *   x_scale       per-tensor activation scale, finite and > 0 (ignored by
 *                 SL_EPI_ACC_I32).
 *   epilogue_kind one of sl_epilogue_kind.
 *   out_scale     per-tensor output scale, finite and > 0, for the int8 kinds
 *                 (ignored otherwise).
 *   y_dev         [m_tokens x n_out] device pointer of the kind's element type
 *                 (int32, fp32 or int8); must not overlap x_dev; 16-byte
 *                 aligned for int32/fp32 output, 4-byte aligned for int8
 *                 (else SL_ERR_INVALID_ARG).
 *   hip_stream    a hipStream_t (NULL = the legacy default stream).
 * The caller keeps X and Y alive until the stream has passed the call.
 * Host cost: the first SL_EPI_I8_GELU run at a given out_scale builds that
 * scale's GELU step table on the host (under 1 ms of one core, typically;
 * up to about 50 ms where it checks every fp32 value of a cell; under a
 * lock that serialises concurrent first uses); the library keeps the 32 most
 * recently built tables in static storage and rebuilds one that has been
 * displaced. No other run allocates or builds anything on the host.
 */
sl_status sparse_linear_run(const sl_packed_weight *w, const int8_t *x_dev, int64_t m_tokens,
                            float x_scale, int32_t epilogue_kind, float out_scale, void *y_dev,
                            void *hip_stream);

/*
 * sparse_linear_run with explicit activation layouts (sl_layout):
 *   x_layout      layout of x_dev (rows = m_tokens, cols = k_in). For
 *                 SL_LAYOUT_T16X32 x_dev must be 16-byte aligned.
 *   y_layout      layout of y_dev (rows = m_tokens, cols = n_out).
 *                 SL_LAYOUT_T16X32 only for SL_EPI_I8 / SL_EPI_I8_GELU, with
 *                 y_dev 16-byte aligned; it writes every real (token,
 *                 channel) byte, padding bytes are left unspecified.
 * Other arguments, results and errors as sparse_linear_run, which is this
 * call with both layouts SL_LAYOUT_ROWS. Bad layout values or alignment:
 * SL_ERR_INVALID_ARG.
 */
sl_status sparse_linear_run_layout(const sl_packed_weight *w, const int8_t *x_dev, int32_t x_layout,
                                   int64_t m_tokens, float x_scale, int32_t epilogue_kind, float out_scale,
                                   void *y_dev, int32_t y_layout, void *hip_stream);

/*
 * Per-tensor symmetric activation quantisation for the first op of a chain
 * (Section "Post-training quantization"): q = clamp(rint(x * (1/scale)), -127, 127)
 * with fl(1/scale) computed once in fp32. Asynchronous on hip_stream.
 *   x_dev  [numel] fp32 device pointer, finite values (non-finite: unspecified q)
 *   numel  >= 0 (0 is a no-op)
 *   scale  finite and > 0
 *   q_dev  [numel] int8 device pointer, must not overlap x_dev
 */
sl_status quantize_act(const float *x_dev, int64_t numel, float scale, int8_t *q_dev, void *hip_stream);

/*
 * quantize_act of a [rows x cols] fp32 row-major tensor into q_layout
 * (sl_layout). SL_LAYOUT_ROWS is quantize_act of rows * cols elements; for
 * SL_LAYOUT_T16X32 q_dev (16-byte aligned) receives ceil(rows/16) *
 * ceil(cols/32) * 512 bytes, padding bytes written as 0. rows, cols >= 0
 * (either 0: no-op); x_dev 4-byte aligned.
 */
sl_status quantize_act_layout(const float *x_dev, int64_t rows, int32_t cols, float scale, int8_t *q_dev,
                              int32_t q_layout, void *hip_stream);

/* Rebuild the dense [n_out x k_in] int8 weight from the handle's GPU tile
 * image (host mirror), into caller memory w_host. Round trip of the packer. */
sl_status sparse_linear_unpack(const sl_packed_weight *w, int8_t *w_host);

/* Shape and number of stored 4x1 blocks. Any output pointer may be NULL. */
sl_status sparse_linear_info(const sl_packed_weight *w, int32_t *n_out, int32_t *k_in, int64_t *nnz_blocks);

/*
 * Copy out the canonical block-sparse (BSR, 4x1 blocks) form:
 *   row_ptr [n_out/4 + 1] uint32: blocks of block-row g are row_ptr[g] .. row_ptr[g+1]-1
 *   col     [nnz_blocks]  uint16: input column of each block, ascending per block-row
 *   vals    [nnz_blocks * 4] int8: W[4g+0..3][col] of each block
 * Buffers are the caller's, sized from sparse_linear_info. Any may be NULL.
 */
sl_status sparse_linear_export_bsr(const sl_packed_weight *w, uint32_t *row_ptr, uint16_t *col, int8_t *vals);

/*
 * Statistics of the GPU tile image: n_tiles channel tiles of 16 output
 * channels; n_entries = matrix-core instructions issued per 16 tokens over all
 * tiles (one per 128-column window that holds a stored block of the tile, plus
 * one per window where some block-row stores 3 or 4 blocks in one aligned
 * group of 4 columns); n_overflow = the latter; image_bytes = bytes of the
 * device image. Any pointer may be NULL.
 */
sl_status sparse_linear_tile_stats(const sl_packed_weight *w, int32_t *n_tiles, int64_t *n_entries,
                                   int64_t *n_overflow, int64_t *image_bytes);

/* Free a handle and its device memory (synchronous). NULL is a no-op. */
void sparse_linear_free(sl_packed_weight *w);

/* Static text for a status code. */
const char *sl_status_string(int32_t status);

/* Thread-local text describing the last failure on this thread ("" if none). */
const char *sl_last_error(void);

/* SL_ABI_VERSION of the loaded library. */
int32_t sl_abi_version(void);

/*
 * Thread-local text naming the kernel and workgroup shape of the last
 * successful sparse_linear_run / sparse_linear_run_layout on this thread
 * ("" before the first): "split st,nt kw=K wpw=W" (split reduction, for
 * few tokens), "panel nt,st,nwv,r" (weight-stationary), "direct st,nt,wm,d"
 * or "staged st,ct,wm,wn,d", followed by " gelu=erf" when an
 * int8 GELU epilogue evaluated erf because its output scale (below about
 * 0.015) admits no step table. For tests and tuning; the text is valid until
 * the next run on this thread.
 */
const char *sl_last_path(void);

/*
 * Kernel selection overrides, for tuning and tests: SL_PATH (split, panel,
 * direct, staged), the tile shapes SL_TILE / SL_DTILE / SL_PTILE and the
 * weight-stationary kernel's token-slice count SL_PSLICES are read from
 * the environment once, at the first run; sl_reload_env() reads
 * them again (call it after changing them, with no run in flight on any
 * thread).
 */
void sl_reload_env(void);

/*
 * Host evaluation of the step table that SL_EPI_I8_GELU runs use in place of
 * erf (Appendix "Graph optimization": GELU fused into the InnerProduct,
 * followed by requantisation as in Section "Sparse GEMM operators"):
 * q[i] = the table's code for the dequantised value y[i] at this out_scale,
 * looked up exactly as the kernels look it up. Host pointers, n >= 0.
 * Returns SL_ERR_UNSUPPORTED when out_scale admits no table (the kernels
 * then evaluate erf), SL_ERR_INVALID_ARG for a bad scale or NULL pointers.
 * For tests of the table against the definition.
 */
sl_status sl_gelu_table_codes(float out_scale, const float *y, int8_t *q, int64_t n);

#ifdef __cplusplus
}
#endif

#endif /* SPARSE_LINEAR_H */
