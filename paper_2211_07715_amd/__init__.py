"""Python binding of the gfx950 sparse INT8 linear library (libsparse_linear.so).

Argument marshalling only: every step of the layer runs in the library's HIP
kernels. PyTorch is used for device memory and streams. There is no CPU or
PyTorch fallback: if the shared library is missing, ``load()`` raises.

    import paper_2211_07715_amd as sl
    pw = sl.PackedWeight.pack(w_int8, w_scale, bias)        # host -> device, once
    q = sl.quantize_act(x_f32_cuda, x_scale)                 # first op of a chain
    y = pw.run(q, x_scale, sl.EPI_I8_GELU, out_scale=so)     # int8 [M, N]

Activations between layers can stay in the 16-token x 32-feature block layout
(LAYOUT_T16X32, 4-D tensors [ceil(M/16), ceil(C/32), 16, 32]), the order the
matrix cores read them in:

    q = sl.quantize_act(x_f32_cuda, x_scale, layout=sl.LAYOUT_T16X32)
    h = pw1.run(q, x_scale, sl.EPI_I8_GELU, out_scale=so, m_tokens=M,
                x_layout=sl.LAYOUT_T16X32, y_layout=sl.LAYOUT_T16X32)
    y = pw2.run(h, so, sl.EPI_F32, m_tokens=M, x_layout=sl.LAYOUT_T16X32)   # fp32 [M, N2]
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsparse_linear.so")

EPI_ACC_I32, EPI_F32, EPI_F32_GELU, EPI_I8, EPI_I8_GELU = 0, 1, 2, 3, 4
EPI_BY_NAME = {"acc_i32": 0, "f32": 1, "f32_gelu": 2, "i8": 3, "i8_gelu": 4}
LAYOUT_ROWS, LAYOUT_T16X32 = 0, 1

SL_OK = 0
STATUS = {0: "SL_OK", -1: "SL_ERR_INVALID_ARG", -2: "SL_ERR_SHAPE", -3: "SL_ERR_HIP", -4: "SL_ERR_OOM",
          -5: "SL_ERR_UNSUPPORTED", -6: "SL_ERR_NOT_ON_DEVICE"}

# every symbol include/sparse_linear.h declares
EXPORTS = ("sparse_linear_pack", "sparse_linear_pack_host", "sparse_linear_run", "sparse_linear_run_layout",
           "quantize_act", "quantize_act_layout",
           "sparse_linear_unpack", "sparse_linear_info", "sparse_linear_export_bsr",
           "sparse_linear_tile_stats", "sparse_linear_free", "sl_status_string", "sl_last_error",
           "sl_abi_version", "sl_last_path", "sl_reload_env", "sl_gelu_table_codes")

# kernel-selection overrides the library reads from the environment
ENV_KEYS = ("SL_PATH", "SL_TILE", "SL_DTILE", "SL_PTILE", "SL_PSLICES")
_env_seen: Optional[tuple] = None

_lib: Optional[ctypes.CDLL] = None


class SparseLinearError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: {STATUS.get(status, status)}: {detail}")
        self.status = status


def load() -> ctypes.CDLL:
    """Load the in-tree shared library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2211_07715_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    pp = ctypes.POINTER(ctypes.c_void_p)
    lib.sparse_linear_pack.argtypes = [vp, i32, i32, i32, i32, vp, vp, pp]
    lib.sparse_linear_pack_host.argtypes = [vp, i32, i32, i32, i32, vp, vp, pp]
    lib.sparse_linear_run.argtypes = [vp, vp, i64, f32, i32, f32, vp, vp]
    lib.sparse_linear_run_layout.argtypes = [vp, vp, i32, i64, f32, i32, f32, vp, i32, vp]
    lib.quantize_act.argtypes = [vp, i64, f32, vp, vp]
    lib.quantize_act_layout.argtypes = [vp, i64, i32, f32, vp, i32, vp]
    lib.sparse_linear_unpack.argtypes = [vp, vp]
    lib.sparse_linear_info.argtypes = [vp, vp, vp, vp]
    lib.sparse_linear_export_bsr.argtypes = [vp, vp, vp, vp]
    lib.sparse_linear_tile_stats.argtypes = [vp, vp, vp, vp, vp]
    for name in ("sparse_linear_pack", "sparse_linear_pack_host", "sparse_linear_run", "sparse_linear_run_layout",
                 "quantize_act", "quantize_act_layout",
                 "sparse_linear_unpack", "sparse_linear_info", "sparse_linear_export_bsr",
                 "sparse_linear_tile_stats"):
        getattr(lib, name).restype = i32
    lib.sparse_linear_free.argtypes = [vp]
    lib.sparse_linear_free.restype = None
    lib.sl_status_string.argtypes = [i32]
    lib.sl_status_string.restype = ctypes.c_char_p
    lib.sl_last_error.argtypes = []
    lib.sl_last_error.restype = ctypes.c_char_p
    lib.sl_abi_version.argtypes = []
    lib.sl_abi_version.restype = i32
    lib.sl_last_path.argtypes = []
    lib.sl_last_path.restype = ctypes.c_char_p
    lib.sl_reload_env.argtypes = []
    lib.sl_reload_env.restype = None
    lib.sl_gelu_table_codes.argtypes = [f32, vp, vp, i64]
    lib.sl_gelu_table_codes.restype = i32
    _lib = lib
    return lib


def _sync_env(lib: ctypes.CDLL):
    """The library reads SL_PATH / SL_*TILE once; have it read them again when
    this process has changed them since the last run."""
    global _env_seen
    now = tuple(os.environ.get(k) for k in ENV_KEYS)
    if now != _env_seen:
        lib.sl_reload_env()
        _env_seen = now


def _check(status: int, where: str):
    if status != SL_OK:
        detail = load().sl_last_error().decode(errors="replace")
        raise SparseLinearError(status, where, detail)


def _np_ptr(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def t16x32_shape(rows: int, cols: int):
    """Shape of a [rows x cols] activation in LAYOUT_T16X32."""
    return ((rows + 15) // 16, (cols + 31) // 32, 16, 32)


def to_t16x32(a: np.ndarray, fill: int = 0) -> np.ndarray:
    """Host copy of an int8 [rows x cols] array in LAYOUT_T16X32 (padding = fill)."""
    rows, cols = a.shape
    rb, cb, _, _ = t16x32_shape(rows, cols)
    p = np.full((rb * 16, cb * 32), fill, dtype=a.dtype)
    p[:rows, :cols] = a
    return np.ascontiguousarray(p.reshape(rb, 16, cb, 32).transpose(0, 2, 1, 3))


def from_t16x32(b: np.ndarray, rows: int, cols: int) -> np.ndarray:
    """The [rows x cols] array held by a LAYOUT_T16X32 array (padding dropped)."""
    rb, cb, _, _ = b.shape
    return np.ascontiguousarray(b.transpose(0, 2, 1, 3).reshape(rb * 16, cb * 32)[:rows, :cols])


def _stream_ptr(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class PackedWeight:
    """An immutable packed 4x1 block-sparse int8 weight (one C handle)."""

    def __init__(self, handle: int, n_out: int, k_in: int, on_device: bool):
        self._h = ctypes.c_void_p(handle)
        self.n_out = n_out
        self.k_in = k_in
        self.on_device = on_device

    @classmethod
    def pack(cls, w: np.ndarray, w_scale: np.ndarray, bias: Optional[np.ndarray] = None,
             host_only: bool = False) -> "PackedWeight":
        lib = load()
        w = np.ascontiguousarray(w, dtype=np.int8)
        if w.ndim != 2:
            raise ValueError("w must be [n_out, k_in]")
        sw = np.ascontiguousarray(w_scale, dtype=np.float32)
        b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
        n, k = w.shape
        if sw.shape != (n,) or (b is not None and b.shape != (n,)):
            raise ValueError("w_scale and bias must have shape [n_out]")
        h = ctypes.c_void_p()
        fn = lib.sparse_linear_pack_host if host_only else lib.sparse_linear_pack
        _check(fn(_np_ptr(w), n, k, 4, 1, _np_ptr(sw), _np_ptr(b), ctypes.byref(h)), fn.__name__)
        return cls(h.value, n, k, not host_only)

    @property
    def handle(self) -> ctypes.c_void_p:
        if not self._h:
            raise ValueError("packed weight was freed")
        return self._h

    def free(self):
        if self._h:
            load().sparse_linear_free(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass

    def info(self):
        n, k, nnzb = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int64()
        _check(load().sparse_linear_info(self.handle, ctypes.byref(n), ctypes.byref(k), ctypes.byref(nnzb)),
               "sparse_linear_info")
        return n.value, k.value, nnzb.value

    def nnz_blocks(self) -> int:
        return self.info()[2]

    def unpack(self) -> np.ndarray:
        out = np.empty((self.n_out, self.k_in), dtype=np.int8)
        _check(load().sparse_linear_unpack(self.handle, _np_ptr(out)), "sparse_linear_unpack")
        return out

    def export_bsr(self):
        nnzb = self.nnz_blocks()
        row_ptr = np.empty(self.n_out // 4 + 1, dtype=np.uint32)
        col = np.empty(nnzb, dtype=np.uint16)
        vals = np.empty((nnzb, 4), dtype=np.int8)
        _check(load().sparse_linear_export_bsr(self.handle, _np_ptr(row_ptr), _np_ptr(col), _np_ptr(vals)),
               "sparse_linear_export_bsr")
        return row_ptr, col, vals

    def tile_stats(self):
        nt, ne, no, ib = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(load().sparse_linear_tile_stats(self.handle, ctypes.byref(nt), ctypes.byref(ne), ctypes.byref(no),
                                               ctypes.byref(ib)), "sparse_linear_tile_stats")
        return {"n_tiles": nt.value, "n_entries": ne.value, "n_overflow": no.value, "image_bytes": ib.value}

    def run(self, x, x_scale: float, kind: int, out_scale: float = 1.0, out=None, stream=None,
            x_layout: int = LAYOUT_ROWS, y_layout: int = LAYOUT_ROWS, m_tokens: Optional[int] = None):
        """Y = epilogue(X W^T) for a CUDA int8 tensor x; returns Y.

        x: [M, k_in] (LAYOUT_ROWS) or t16x32_shape(M, k_in) with m_tokens=M
        (LAYOUT_T16X32). Y: [M, n_out] of the kind's dtype, or, for the int8
        kinds with y_layout=LAYOUT_T16X32, t16x32_shape(M, n_out) int8."""
        import torch
        if x.dtype != torch.int8 or not x.is_cuda or not x.is_contiguous():
            raise ValueError("x must be a contiguous CUDA int8 tensor")
        if x_layout == LAYOUT_ROWS:
            if x.dim() != 2 or x.shape[1] != self.k_in:
                raise ValueError(f"x must be [M, {self.k_in}]")
            m = x.shape[0] if m_tokens is None else int(m_tokens)
            if m != x.shape[0]:
                raise ValueError("m_tokens differs from x's rows")
        elif x_layout == LAYOUT_T16X32:
            if m_tokens is None:
                raise ValueError("m_tokens is required with LAYOUT_T16X32 input")
            m = int(m_tokens)
            if tuple(x.shape) != t16x32_shape(m, self.k_in):
                raise ValueError(f"x must have shape {t16x32_shape(m, self.k_in)}")
        else:
            raise ValueError(f"unknown x_layout {x_layout}")
        dt = {EPI_ACC_I32: torch.int32, EPI_F32: torch.float32, EPI_F32_GELU: torch.float32,
              EPI_I8: torch.int8, EPI_I8_GELU: torch.int8}[kind]
        shape = t16x32_shape(m, self.n_out) if y_layout == LAYOUT_T16X32 else (m, self.n_out)
        if out is None:
            out = torch.empty(shape, dtype=dt, device=x.device)
        elif out.dtype != dt or tuple(out.shape) != tuple(shape) or not out.is_contiguous():
            raise ValueError("out has the wrong dtype/shape or is not contiguous")
        lib = load()
        _sync_env(lib)
        _check(lib.sparse_linear_run_layout(self.handle, ctypes.c_void_p(x.data_ptr()), int(x_layout), m,
                                               float(x_scale), int(kind), float(out_scale),
                                               ctypes.c_void_p(out.data_ptr()), int(y_layout), _stream_ptr(stream)),
               "sparse_linear_run_layout")
        return out


def last_path() -> str:
    """Kernel and workgroup shape of the last successful run on this thread."""
    return load().sl_last_path().decode()


def gelu_table_codes(out_scale: float, y: np.ndarray) -> Optional[np.ndarray]:
    """int8 codes of the GELU + requantisation step table for fp32 values y,
    looked up as the kernels do; None when out_scale admits no table."""
    lib = load()
    y = np.ascontiguousarray(y, dtype=np.float32)
    q = np.empty(y.shape, dtype=np.int8)
    st = lib.sl_gelu_table_codes(float(out_scale), _np_ptr(y), _np_ptr(q), y.size)
    if st == -5:
        return None
    _check(st, "sl_gelu_table_codes")
    return q


def quantize_act(x, scale: float, out=None, stream=None, layout: int = LAYOUT_ROWS):
    """q = clamp(rint(x / scale), -127, 127) for a contiguous CUDA fp32 tensor:
    same shape (LAYOUT_ROWS), or, for a 2-D x [rows, cols] and
    layout=LAYOUT_T16X32, int8 of shape t16x32_shape(rows, cols)."""
    import torch
    if x.dtype != torch.float32 or not x.is_cuda or not x.is_contiguous():
        raise ValueError("x must be a contiguous CUDA float32 tensor")
    if layout == LAYOUT_ROWS:
        if out is None:
            out = torch.empty(x.shape, dtype=torch.int8, device=x.device)
        elif out.dtype != torch.int8 or out.numel() != x.numel() or not out.is_contiguous():
            raise ValueError("out must be a contiguous int8 tensor with x's size")
        _check(load().quantize_act(ctypes.c_void_p(x.data_ptr()), x.numel(), float(scale),
                                   ctypes.c_void_p(out.data_ptr()), _stream_ptr(stream)), "quantize_act")
        return out
    if layout != LAYOUT_T16X32 or x.dim() != 2:
        raise ValueError("LAYOUT_T16X32 quantisation takes a 2-D x [rows, cols]")
    rows, cols = x.shape
    shape = t16x32_shape(rows, cols)
    if out is None:
        out = torch.empty(shape, dtype=torch.int8, device=x.device)
    elif out.dtype != torch.int8 or tuple(out.shape) != shape or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous int8 tensor of shape {shape}")
    _check(load().quantize_act_layout(ctypes.c_void_p(x.data_ptr()), rows, cols, float(scale),
                                      ctypes.c_void_p(out.data_ptr()), int(layout), _stream_ptr(stream)),
           "quantize_act_layout")
    return out
