"""GPU parity of the 16-token x 32-feature block activation layout
(SL_LAYOUT_T16X32) against the CPU oracle, which works on row-major arrays;
the layout conversions are the host helpers pinned in test_pack_host.py.

Bars as in test_gpu_parity.py: int32 bit-exact, fp32 max|err| <= 1e-5 *
max|ref|, int8 within 1 LSB in at most 0.01 % of the elements. The padding of
a block-layout input is filled with junk (99): the header promises it never
reaches a stored output.
"""
import numpy as np
import pytest

import oracle
import oracle.chain as ochain
import workloads as wk
from test_gpu_parity import KINDS, _calib, _case, check, say

pytestmark = pytest.mark.gpu

T = 1  # SL_LAYOUT_T16X32


def _to_dev(hip, a_blocks):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a_blocks)).cuda()


def _so_for(kind, x, w, sw, b):
    if kind not in (3, 4):
        return 1.0
    g = oracle.linear(x, w, 0.02, sw, b, 1 if kind == 3 else 2)
    return float(oracle.calibrate_out_scale(g)) or 1.0


# 36 and 160 columns end in a partial block (padding features); 49152 x 768
# makes the persistent grid loop over its pieces
@pytest.mark.parametrize("rows,cols", [(1, 1), (16, 32), (17, 33), (5, 100), (3, 4), (31, 160), (48, 36),
                                       (300, 768), (33, 3072), (4096, 768), (49152, 768)])
def test_quantize_act_t16x32(hip, rows, cols):
    import torch
    rng = np.random.default_rng(rows + 7 * cols)
    x = (rng.standard_normal((rows, cols)) * 3.0).astype(np.float32)
    say(f"quantize t16x32 rows={rows} cols={cols}")
    ref = oracle.quantize(x, 0.02)
    xd = torch.from_numpy(x).cuda()
    q = hip.quantize_act(xd, 0.02, layout=T)
    torch.cuda.synchronize()
    qb = q.cpu().numpy()
    assert qb.shape == hip.t16x32_shape(rows, cols)
    assert np.array_equal(hip.from_t16x32(qb, rows, cols), ref)
    # padding is written as zeros
    assert np.array_equal(qb, hip.to_t16x32(ref, fill=0))
    if cols % 4 == 0 and rows > 1:  # misaligned source rows: the scalar path
        big = torch.zeros(rows * cols + 1, dtype=torch.float32, device="cuda")
        big[1:].copy_(xd.reshape(-1))
        q2 = hip.quantize_act(big[1:].view(rows, cols), 0.02, layout=T)
        torch.cuda.synchronize()
        assert np.array_equal(q2.cpu().numpy(), qb)


SHAPES = [(1, 4, 32), (16, 16, 64), (17, 20, 100), (64, 48, 768), (65, 768, 768), (200, 64, 1025), (33, 32, 3072),
          (130, 1024, 4096), (5, 12, 2049), (300, 3072, 768)]


@pytest.mark.parametrize("m,n,k", SHAPES)
@pytest.mark.parametrize("x_layout,y_layout", [(T, 0), (T, T), (0, T)])
def test_block_layout_all_kinds(hip, m, n, k, x_layout, y_layout):
    import torch
    w, sw, b, rng = _case(n, k, 0.3, 31 * m + 7 * n + k)
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    say(f"layout m={m} n={n} k={k} x_layout={x_layout} y_layout={y_layout}")
    pw = hip.PackedWeight.pack(w, sw, b)
    xd = _to_dev(hip, hip.to_t16x32(x, fill=99)) if x_layout == T else torch.from_numpy(x).cuda()
    for name, kind in KINDS.items():
        if y_layout == T and kind not in (3, 4):
            continue
        so = _so_for(kind, x, w, sw, b)
        ref = oracle.linear(x, w, 0.02, sw, b, kind, so=so)
        y = pw.run(xd, 0.02, kind, out_scale=so, x_layout=x_layout, y_layout=y_layout, m_tokens=m)
        torch.cuda.synchronize()
        got = y.cpu().numpy()
        if y_layout == T:
            got = hip.from_t16x32(got, m, n)
        check(kind, got, ref, f"{name} m={m} n={n} k={k} layouts=({x_layout},{y_layout})")
    pw.free()


@pytest.mark.parametrize("dtile", ["2,6,4,4", "1,6,4,6", "1,2,4,8"])
def test_block_layout_each_shape(hip, monkeypatch, dtile):
    import torch
    monkeypatch.setenv("SL_PATH", "direct")
    monkeypatch.setenv("SL_DTILE", dtile)
    for (m, n, k) in [(77, 96, 768), (300, 200, 1000), (16, 3072, 768)]:
        w, sw, b, rng = _case(n, k, 0.15, m + n + k)
        x = rng.integers(-127, 128, (m, k), dtype=np.int8)
        say(f"layout shape {dtile} m={m} n={n} k={k}")
        pw = hip.PackedWeight.pack(w, sw, b)
        xd = _to_dev(hip, hip.to_t16x32(x, fill=-5))
        for kind in (0, 4):
            so = _so_for(kind, x, w, sw, b)
            ref = oracle.linear(x, w, 0.02, sw, b, kind, so=so)
            yl = T if kind == 4 else 0
            y = pw.run(xd, 0.02, kind, out_scale=so, x_layout=T, y_layout=yl, m_tokens=m)
            torch.cuda.synchronize()
            got = y.cpu().numpy()
            check(kind, hip.from_t16x32(got, m, n) if yl == T else got, ref, f"{dtile} kind={kind}")
        pw.free()


def test_block_layout_rejections(hip):
    import ctypes
    import torch
    w, sw, b, rng = _case(16, 64, 0.3, 9)
    pw = hip.PackedWeight.pack(w, sw, b)
    lib = hip.load()
    x = torch.zeros(hip.t16x32_shape(4, 64), dtype=torch.int8, device="cuda")
    yf = torch.zeros((4, 16), dtype=torch.float32, device="cuda")
    y8 = torch.zeros(hip.t16x32_shape(4, 16), dtype=torch.int8, device="cuda")
    xp, yfp, y8p = (ctypes.c_void_p(t.data_ptr()) for t in (x, yf, y8))
    # block-layout output only for the int8 kinds
    assert lib.sparse_linear_run_layout(pw.handle, xp, T, 4, 0.02, 1, 1.0, yfp, T, None) == -1
    # unknown layouts
    assert lib.sparse_linear_run_layout(pw.handle, xp, 2, 4, 0.02, 3, 1.0, y8p, 0, None) == -1
    assert lib.sparse_linear_run_layout(pw.handle, xp, T, 4, 0.02, 3, 1.0, y8p, 5, None) == -1
    # 16-byte alignment of block-layout tensors
    assert lib.sparse_linear_run_layout(pw.handle, ctypes.c_void_p(x.data_ptr() + 4), T, 4, 0.02, 3, 1.0, y8p, T,
                                        None) == -1
    assert lib.sparse_linear_run_layout(pw.handle, xp, T, 4, 0.02, 3, 1.0, ctypes.c_void_p(y8.data_ptr() + 4), T,
                                        None) == -1
    assert lib.sparse_linear_run_layout(pw.handle, xp, T, 4, 0.02, 3, 1.0, y8p, T, None) == 0
    torch.cuda.synchronize()
    pw.free()


@pytest.mark.parametrize("name", ["c1", "c2", "c3_seq128_s80"])
def test_chain_in_block_layout(hip, name):
    """A workload's layer chain with every activation in the block layout: the
    first op's input is quantised on the GPU straight into it, int8 outputs
    are written in it, and each op reads the oracle's input for that op in it
    (so an int8 rounding difference allowed by the bar does not compound)."""
    import torch
    wl = wk.workloads()[name]
    calib = _calib()[name]
    outs, scales, ins = ochain.run(wl, calib=calib)
    for layer, op in wk.op_list(wl):
        key = ochain.op_key(layer, op.name)
        src = wl.op_src(layer, op)
        kind = KINDS[wl.op_kind(layer, op)]
        so = float(calib.get(key, 1.0))
        x_ref, sx = ins[key]
        if src == "seeded":  # quantise the fp32 values the oracle's int8 input came from
            xf = (x_ref.astype(np.float32) * np.float32(sx)).astype(np.float32)
            assert np.array_equal(oracle.quantize(xf, sx), x_ref)
            xd = hip.quantize_act(torch.from_numpy(xf).cuda(), sx, layout=T)
        else:
            xd = _to_dev(hip, hip.to_t16x32(x_ref, fill=77))
        wd = wk.op_weight(wl, layer, op)
        pw = hip.PackedWeight.pack(wd["w"], wd["sw"], wd["b"])
        yl = T if kind in (3, 4) else 0
        say(f"{name} {key} kind={kind} block layout in, layout {yl} out")
        y = pw.run(xd, sx, kind, out_scale=so, x_layout=T, y_layout=yl, m_tokens=wl.m)
        torch.cuda.synchronize()
        got = y.cpu().numpy()
        if yl == T:
            got = hip.from_t16x32(got, wl.m, op.n_out)
        check(kind, got, outs[key], f"{name} {key}")
        pw.free()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["c4", "c4_bertl"])
def test_full_size_chain_in_block_layout(hip, name):
    """M = 49152 tokens, every row of every op: each op reads the oracle's own
    input for it (the chained int8 output of the op before, or its seeded
    input) in the block layout, int8 outputs are written in it, and the int32
    accumulators of every op are compared too, bit for bit."""
    import torch
    wl = wk.workloads()[name]
    calib = _calib()[name]
    for key, wd, x, sx, kind, so, acc, ref in ochain.steps(wl, calib):
        n_out, k_in = wd["w"].shape
        say(f"{name} {key} kind={kind} m={wl.m} n={n_out} k={k_in}: every row, block layout")
        pw = hip.PackedWeight.pack(wd["w"], wd["sw"], wd["b"])
        xd = _to_dev(hip, hip.to_t16x32(x, fill=77))
        yl = T if kind in (3, 4) else 0
        y = pw.run(xd, sx, kind, out_scale=so, x_layout=T, y_layout=yl, m_tokens=wl.m)
        torch.cuda.synchronize()
        got = y.cpu().numpy()
        del y
        if yl == T:
            got = hip.from_t16x32(got, wl.m, n_out)
        check(kind, got, ref, f"{name} {key}")
        del got
        a = pw.run(xd, sx, 0, x_layout=T, m_tokens=wl.m)
        torch.cuda.synchronize()
        check(0, a.cpu().numpy(), acc, f"{name} {key} int32")
        del a, xd
        pw.free()


@pytest.mark.parametrize("name", ["c1", "c2"])
def test_chain_gpu_to_gpu(hip, name):
    """The whole chain on the GPU: the first op's input is quantised on the
    GPU into the block layout, and every later op reads the previous op's
    int8 output where the GPU wrote it (nothing returns to the host between
    ops). Each hop's input is held to the int8 bar against the oracle chain's
    input for that op, and each hop's output to its kind's bar against the
    oracle applied to the very input the hop consumed."""
    import torch
    wl = wk.workloads()[name]
    calib = _calib()[name]
    outs, scales, ins = ochain.run(wl, calib=calib)
    dev = {}
    for layer, op in wk.op_list(wl):
        key = ochain.op_key(layer, op.name)
        src = wl.op_src(layer, op)
        kind = KINDS[wl.op_kind(layer, op)]
        so = float(calib.get(key, 1.0))
        x_ref, sx = ins[key]
        if src == "seeded":
            xf = (x_ref.astype(np.float32) * np.float32(sx)).astype(np.float32)
            xd = hip.quantize_act(torch.from_numpy(xf).cuda(), sx, layout=T)
        else:
            xd = dev[src]
        wd = wk.op_weight(wl, layer, op)
        pw = hip.PackedWeight.pack(wd["w"], wd["sw"], wd["b"])
        yl = T if kind in (3, 4) else 0
        say(f"{name} {key} kind={kind}: input from {src} on the GPU")
        y = pw.run(xd, sx, kind, out_scale=so, x_layout=T, y_layout=yl, m_tokens=wl.m)
        dev[key] = y
        torch.cuda.synchronize()
        x_used = hip.from_t16x32(xd.cpu().numpy(), wl.m, op.k_in)
        check(3, x_used, x_ref, f"{name} {key}: hop input vs the oracle chain")
        got = y.cpu().numpy()
        if yl == T:
            got = hip.from_t16x32(got, wl.m, op.n_out)
        ref = oracle.linear(x_used, wd["w"], sx, wd["sw"], wd["b"], kind, so=so)
        check(kind, got, ref, f"{name} {key}: hop output")
        pw.free()
