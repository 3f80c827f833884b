"""Host-side tests of the C-ABI library (no GPU needed).

* the shared library loads and exports every symbol include/sparse_linear.h declares;
* the packer's canonical BSR form and its GPU tile image both round-trip to
  the dense weight, across sparsities, ragged shapes and chunked K;
* argument validation returns the documented status codes.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2211_07715_amd as sl
from workloads import make_weight, random_block_sparse

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_symbols():
    with open(os.path.join(ROOT, "include", "sparse_linear.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", text)) - {"if", "sizeof"}


def test_library_exports_every_declared_symbol():
    lib = sl.load()
    declared = _header_symbols()
    assert declared == set(sl.EXPORTS), declared ^ set(sl.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name
    assert lib.sl_abi_version() == 3
    assert lib.sl_status_string(-2) == b"SL_ERR_SHAPE"


def test_library_has_no_cpu_fallback_symbols():
    # the product library links no oracle code
    lib = sl.load()
    for name in ("oracle_linear", "oracle_acc", "oracle_quantize"):
        with pytest.raises(AttributeError):
            getattr(lib, name)


def _bsr_reference(w):
    n, k = w.shape
    blocks = w.reshape(n // 4, 4, k)
    keep = np.any(blocks != 0, axis=1)  # [n/4, k]
    row_ptr = np.concatenate([[0], np.cumsum(keep.sum(axis=1))]).astype(np.uint32)
    g, c = np.nonzero(keep)
    vals = blocks[g, :, c]
    return row_ptr, c.astype(np.uint16), vals


@pytest.mark.parametrize("n,k,density", [(4, 1, 1.0), (4, 7, 0.5), (16, 64, 0.3), (20, 33, 0.6), (768, 768, 0.2),
                                         (3072, 768, 0.1), (768, 3072, 0.1), (64, 1500, 0.25), (8, 2049, 0.05),
                                         (28, 100, 0.0), (12, 64, 1.0)])
def test_pack_roundtrip(n, k, density):
    rng = np.random.default_rng(n * 7 + k)
    w = random_block_sparse(n, k, density, rng)
    # a stored block may hold zeros; an all-zero surviving block is dropped
    sw = rng.uniform(0.001, 0.01, n).astype(np.float32)
    pw = sl.PackedWeight.pack(w, sw, None, host_only=True)
    assert np.array_equal(pw.unpack(), w)
    row_ptr, col, vals = pw.export_bsr()
    r2, c2, v2 = _bsr_reference(w)
    assert np.array_equal(row_ptr, r2)
    assert np.array_equal(col, c2)
    assert np.array_equal(vals, v2)
    n2, k2, nnzb = pw.info()
    assert (n2, k2, nnzb) == (n, k, int(r2[-1]))
    st = pw.tile_stats()
    assert st["n_tiles"] == (n + 15) // 16
    assert 0 <= st["n_overflow"] <= st["n_entries"]
    _check_entry_counts(w, st)
    pw.free()


def _check_entry_counts(w, st):
    """Entries = one per (16-channel tile, 128-column window) holding a stored
    block, plus one where a block-row stores 3-4 blocks in an aligned group of
    4 columns (the 4:2 instruction takes at most 2 per group)."""
    n, k = w.shape
    keep = np.any(w.reshape(n // 4, 4, k) != 0, axis=1)          # [brows, k]
    nbr = n // 4
    kp = (k + 127) // 128 * 128
    kk = np.zeros((nbr, kp), bool)
    kk[:, :k] = keep
    per_group = kk.reshape(nbr, kp // 4, 4).sum(axis=2)          # [brows, groups]
    nt = (n + 15) // 16
    pad_rows = nt * 4 - nbr
    kk = np.concatenate([kk, np.zeros((pad_rows, kp), bool)])
    per_group = np.concatenate([per_group, np.zeros((pad_rows, kp // 4), per_group.dtype)])
    win_any = kk.reshape(nt, 4, kp // 128, 128).any(axis=(1, 3))
    win_ovf = (per_group.reshape(nt, 4, kp // 128, 32) > 2).any(axis=(1, 3))
    assert st["n_entries"] == int(win_any.sum() + win_ovf.sum())
    assert st["n_overflow"] == int(win_ovf.sum())


def test_pack_entry_statistics_match_mask():
    wd = make_weight(3072, 768, 0.9, seed=0, cfg=1, op=2)
    pw = sl.PackedWeight.pack(wd["w"], wd["sw"], wd["b"], host_only=True)
    st = pw.tile_stats()
    _check_entry_counts(wd["w"], st)
    # at 10 % block density about a third of the (tile, window) pairs overflow
    assert 0.25 < st["n_overflow"] / (st["n_entries"] - st["n_overflow"]) < 0.5


def test_pack_dense_groups_need_overflow():
    # a block-row with all 4 blocks of a group stored needs the overflow entry
    w = np.zeros((16, 8), np.int8)
    w[0:4, 0:4] = np.arange(1, 17, dtype=np.int8).reshape(4, 4)
    w[4:8, 5] = 7
    pw = sl.PackedWeight.pack(w, np.ones(16, np.float32), host_only=True)
    st = pw.tile_stats()
    assert (st["n_entries"], st["n_overflow"]) == (2, 1)
    assert np.array_equal(pw.unpack(), w)


def test_pack_zero_blocks_inside_stored_blocks():
    w = np.zeros((8, 5), np.int8)
    w[0, 1] = 3      # block (0, 1) stored, 3 of its values zero
    w[7, 4] = -127   # block (1, 4)
    pw = sl.PackedWeight.pack(w, np.ones(8, np.float32), host_only=True)
    assert pw.nnz_blocks() == 2
    row_ptr, col, vals = pw.export_bsr()
    assert list(row_ptr) == [0, 1, 2] and list(col) == [1, 4]
    assert vals.tolist() == [[3, 0, 0, 0], [0, 0, 0, -127]]
    assert np.array_equal(pw.unpack(), w)


def _raw_pack(w, n, k, bh=4, bw=1, sw=None, bias=None, host=True):
    lib = sl.load()
    h = ctypes.c_void_p()
    fn = lib.sparse_linear_pack_host if host else lib.sparse_linear_pack
    st = fn(None if w is None else ctypes.c_void_p(w.ctypes.data), n, k, bh, bw,
            None if sw is None else ctypes.c_void_p(sw.ctypes.data),
            None if bias is None else ctypes.c_void_p(bias.ctypes.data), ctypes.byref(h))
    return st, h


def test_pack_validation_status_codes():
    w = np.ones((8, 8), np.int8)
    sw = np.ones(8, np.float32)
    assert _raw_pack(w, 8, 8, sw=sw)[0] == 0
    assert _raw_pack(w, 6, 8, sw=sw)[0] == -2          # n_out % 4
    assert _raw_pack(w, 0, 8, sw=sw)[0] == -2
    assert _raw_pack(w, 8, 0, sw=sw)[0] == -2          # k_in < 1
    assert _raw_pack(w, 8, 70000, sw=sw)[0] == -2      # k_in > 65535
    assert _raw_pack(w, 8, 8, bh=2, sw=sw)[0] == -1    # block shape
    assert _raw_pack(w, 8, 8, bw=4, sw=sw)[0] == -1
    assert _raw_pack(None, 8, 8, sw=sw)[0] == -1       # NULL
    assert _raw_pack(w, 8, 8, sw=None)[0] == -1
    bad = sw.copy(); bad[3] = 0.0
    assert _raw_pack(w, 8, 8, sw=bad)[0] == -1         # non-positive scale
    bad[3] = np.nan
    assert _raw_pack(w, 8, 8, sw=bad)[0] == -1
    b = np.zeros(8, np.float32); b[1] = np.inf
    assert _raw_pack(w, 8, 8, sw=sw, bias=b)[0] == -1  # non-finite bias
    st, h = _raw_pack(w, 6, 8, sw=sw)
    assert st == -2 and not h.value                    # *out cleared on failure
    assert b"multiple of 4" in sl.load().sl_last_error()


def test_run_on_host_handle_is_rejected():
    lib = sl.load()
    w = np.ones((8, 8), np.int8)
    pw = sl.PackedWeight.pack(w, np.ones(8, np.float32), host_only=True)
    st = lib.sparse_linear_run(pw.handle, ctypes.c_void_p(16), 4, 1.0, 1, 1.0, ctypes.c_void_p(16), None)
    assert st == -6
    # argument checks happen before any device work
    st = lib.sparse_linear_run(None, None, 4, 1.0, 1, 1.0, None, None)
    assert st == -1
    lib.sparse_linear_free(None)  # NULL is a no-op


def test_quantize_act_argument_checks_without_gpu():
    lib = sl.load()
    assert lib.quantize_act(None, 0, 1.0, None, None) == 0      # empty: no-op
    assert lib.quantize_act(None, -1, 1.0, None, None) == -2
    assert lib.quantize_act(None, 4, 0.0, None, None) == -1
    assert lib.quantize_act(None, 4, float("nan"), None, None) == -1
    assert lib.quantize_act(None, 4, 1.0, None, None) == -1     # NULL buffers


def test_run_layout_argument_checks_without_gpu():
    lib = sl.load()
    w = np.ones((8, 8), np.int8)
    pw = sl.PackedWeight.pack(w, np.ones(8, np.float32), host_only=True)
    p = ctypes.c_void_p(16)
    assert lib.sparse_linear_run_layout(None, p, 0, 4, 1.0, 1, 1.0, p, 0, None) == -1
    assert lib.sparse_linear_run_layout(pw.handle, p, 1, 4, 1.0, 3, 1.0, p, 1, None) == -6
    pw.free()


def test_quantize_act_layout_argument_checks_without_gpu():
    lib = sl.load()
    assert lib.quantize_act_layout(None, 0, 8, 1.0, None, 1, None) == 0      # empty: no-op
    assert lib.quantize_act_layout(None, 4, 0, 1.0, None, 1, None) == 0
    assert lib.quantize_act_layout(None, -1, 8, 1.0, None, 1, None) == -2
    assert lib.quantize_act_layout(None, 4, -8, 1.0, None, 1, None) == -2
    assert lib.quantize_act_layout(None, 4, 8, 1.0, None, 7, None) == -1     # unknown layout
    assert lib.quantize_act_layout(None, 4, 8, 0.0, None, 1, None) == -1
    assert lib.quantize_act_layout(None, 4, 8, 1.0, None, 1, None) == -1     # NULL pointers
    # 16-byte alignment of the block-layout output
    assert lib.quantize_act_layout(ctypes.c_void_p(64), 4, 8, 1.0, ctypes.c_void_p(72), 1, None) == -1


@pytest.mark.parametrize("rows,cols", [(1, 1), (16, 32), (17, 33), (5, 100), (64, 768), (31, 3072)])
def test_t16x32_layout_helpers(rows, cols):
    # the block layout as the header defines it: element (t, c) at byte
    # ((t / 16) * C + c / 32) * 512 + (t % 16) * 32 + c % 32, C = ceil(cols / 32)
    rng = np.random.default_rng(rows * 1000 + cols)
    a = rng.integers(-127, 128, (rows, cols), dtype=np.int8)
    b = sl.to_t16x32(a, fill=99)
    assert b.shape == sl.t16x32_shape(rows, cols)
    flat = b.reshape(-1)
    C = (cols + 31) // 32
    t, c = np.meshgrid(np.arange(rows), np.arange(cols), indexing="ij")
    off = ((t // 16) * C + c // 32) * 512 + (t % 16) * 32 + c % 32
    assert np.array_equal(flat[off], a)
    mask = np.ones(flat.size, bool)
    mask[off.reshape(-1)] = False
    assert (flat[mask] == 99).all()  # everything else is padding
    assert np.array_equal(sl.from_t16x32(b, rows, cols), a)
