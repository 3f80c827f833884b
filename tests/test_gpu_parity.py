"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars (from the layer's definition):
  int32 accumulators     bit-exact
  fp32 outputs           max|err| <= 1e-5 * max|ref|
  requantised int8       |err| <= 1 LSB, in at most 0.01 % of the elements
Every input comes from the seeded generators or from the oracle itself.
"""
import json
import os
import sys

import numpy as np
import pytest

import oracle
import oracle.chain as ochain
import workloads as wk

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
KINDS = {"acc_i32": 0, "f32": 1, "f32_gelu": 2, "i8": 3, "i8_gelu": 4}


def _calib():
    with open(os.path.join(GOLDEN, "calibration.json")) as f:
        return json.load(f)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def check(kind, got, ref, what=""):
    if kind == 0:
        assert got.dtype == np.int32 and np.array_equal(got, ref), f"{what}: int32 mismatch " \
            f"({int((got != ref).sum())} of {ref.size})"
    elif kind in (1, 2):
        scale = float(np.abs(ref).max()) if ref.size else 0.0
        err = float(np.abs(got.astype(np.float64) - ref.astype(np.float64)).max()) if ref.size else 0.0
        assert err <= 1e-5 * scale, f"{what}: fp32 max err {err} > 1e-5 * {scale}"
    else:
        d = np.abs(got.astype(np.int32) - ref.astype(np.int32))
        n_bad = int((d > 0).sum())
        assert d.size == 0 or d.max() <= 1, f"{what}: int8 error {d.max()} LSB"
        assert n_bad <= 1e-4 * d.size, f"{what}: {n_bad} of {d.size} int8 outputs differ by 1 LSB"


def run_gpu(hip, pw, x_np, sx, kind, so=1.0, x_dev=None):
    import torch
    x = torch.from_numpy(np.ascontiguousarray(x_np)).cuda() if x_dev is None else x_dev
    y = pw.run(x, sx, kind, out_scale=so)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def _case(n, k, density, seed):
    rng = np.random.default_rng(seed)
    w = wk.random_block_sparse(n, k, density, rng)
    sw = rng.uniform(0.001, 0.01, n).astype(np.float32)
    b = rng.normal(0, 0.02, n).astype(np.float32)
    return w, sw, b, rng


SMALL = [(1, 4, 1), (3, 16, 7), (16, 16, 64), (17, 20, 100), (64, 48, 768), (65, 768, 768), (200, 64, 1025),
         (33, 32, 3072), (130, 1024, 4096), (5, 12, 2049), (40, 72, 64)]


# kernel paths: the default choice (the split-reduction kernel for few
# aligned token rows, the weight-stationary kernel where it pays, else the
# staged kernel for row-major token rows), the staged and the split-reduction
# kernels forced, and the direct-operand kernel in each of its workgroup
# shapes (the weight-stationary shapes are covered in test_gpu_panel.py)
PATHS = {"default": {}, "staged": {"SL_PATH": "staged"}, "split": {"SL_PATH": "split"},
         "direct": {"SL_PATH": "direct"},
         "direct_64x96": {"SL_PATH": "direct", "SL_DTILE": "1,6,4,6"},
         "direct_64x32": {"SL_PATH": "direct", "SL_DTILE": "1,2,4,8"},
         "direct_128x96": {"SL_PATH": "direct", "SL_DTILE": "2,6,4,4"}}


@pytest.mark.parametrize("m,n,k", SMALL)
@pytest.mark.parametrize("density", [0.0, 0.1, 0.35, 1.0])
@pytest.mark.parametrize("path", list(PATHS))
def test_small_shapes_all_kinds(hip, monkeypatch, m, n, k, density, path):
    if path.startswith("direct_") and density in (0.0, 1.0):
        pytest.skip("the extreme densities run on each kernel's own shape choice")
    for key, val in PATHS[path].items():
        monkeypatch.setenv(key, val)
    w, sw, b, rng = _case(n, k, density, 1000 * m + 10 * n + k + int(density * 100))
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    say(f"small m={m} n={n} k={k} d={density} path={path}")
    pw = hip.PackedWeight.pack(w, sw, b)
    for name, kind in KINDS.items():
        so = 1.0
        if kind in (3, 4):
            g = oracle.linear(x, w, 0.02, sw, b, 1 if kind == 3 else 2)
            so = float(oracle.calibrate_out_scale(g)) or 1.0
        ref = oracle.linear(x, w, 0.02, sw, b, kind, so=so)
        got = run_gpu(hip, pw, x, 0.02, kind, so)
        check(kind, got, ref, f"{name} m={m} n={n} k={k} d={density}")
        if path == "split" and k % 16 == 0:
            assert hip.last_path().startswith("split"), hip.last_path()
    pw.free()


def test_empty_and_degenerate(hip):
    import torch
    w, sw, b, rng = _case(16, 64, 0.3, 5)
    pw = hip.PackedWeight.pack(w, sw, b)
    x = torch.empty((0, 64), dtype=torch.int8, device="cuda")
    y = pw.run(x, 0.02, 1)
    assert y.shape == (0, 16)
    # all-zero weight: outputs are the bias exactly (and GELU / requant of it)
    wz = np.zeros((16, 64), np.int8)
    pz = hip.PackedWeight.pack(wz, sw, b)
    xs = rng.integers(-127, 128, (20, 64), dtype=np.int8)
    assert np.array_equal(run_gpu(hip, pz, xs, 0.02, 1), np.broadcast_to(b, (20, 16)))
    assert not run_gpu(hip, pz, xs, 0.02, 0).any()
    # identity weight reproduces the input
    eye = np.eye(64, dtype=np.int8)
    pe = hip.PackedWeight.pack(eye, np.ones(64, np.float32), None)
    xe = rng.integers(-127, 128, (33, 64), dtype=np.int8)
    assert np.array_equal(run_gpu(hip, pe, xe, 1.0, 0), xe.astype(np.int32))
    assert np.array_equal(run_gpu(hip, pe, xe, 1.0, 3, 1.0), xe)


def test_misaligned_input_view(hip):
    import torch
    w, sw, b, rng = _case(48, 768, 0.2, 6)
    pw = hip.PackedWeight.pack(w, sw, b)
    m = 70
    x = rng.integers(-127, 128, (m, 768), dtype=np.int8)
    big = torch.zeros(m * 768 + 16, dtype=torch.int8, device="cuda")
    view = big[3:3 + m * 768].view(m, 768)
    view.copy_(torch.from_numpy(x).cuda())
    got = run_gpu(hip, pw, x, 0.02, 0, x_dev=view)
    assert np.array_equal(got, oracle.acc(x, w))


def test_bad_output_alignment_is_rejected(hip):
    import ctypes
    import torch
    w, sw, b, rng = _case(16, 64, 0.3, 7)
    pw = hip.PackedWeight.pack(w, sw, b)
    x = torch.zeros((4, 64), dtype=torch.int8, device="cuda")
    y = torch.zeros(4 * 16 + 4, dtype=torch.float32, device="cuda")
    lib = hip.load()
    st = lib.sparse_linear_run(pw.handle, ctypes.c_void_p(x.data_ptr()), 4, 0.02, 1, 1.0,
                               ctypes.c_void_p(y.data_ptr() + 4), None)
    assert st == -1


def test_same_handle_two_streams(hip):
    import torch
    w, sw, b, rng = _case(3072, 768, 0.1, 8)
    pw = hip.PackedWeight.pack(w, sw, b)
    xs = [torch.from_numpy(rng.integers(-127, 128, (1000, 768), dtype=np.int8)).cuda() for _ in range(2)]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = []
    for s, x in zip(streams, xs):
        with torch.cuda.stream(s):
            outs.append(pw.run(x, 0.02, 0, stream=s))
    torch.cuda.synchronize()
    for x, y in zip(xs, outs):
        assert np.array_equal(y.cpu().numpy(), oracle.acc(x.cpu().numpy(), w))


def test_split_reduction_limits(hip, monkeypatch):
    """The split-reduction kernel covers reductions of up to 32 windows
    (k <= 4096): at 32 windows it runs with 16 waves of 2 windows; at 33
    SL_PATH=split falls back to another kernel with the same results. Both
    with the block layout in and out and the int8 GELU epilogue."""
    import torch
    monkeypatch.setenv("SL_PATH", "split")
    for k, want_split in ((4096, True), (4224, False)):
        w, sw, b, rng = _case(96, k, 0.2, k)
        x = rng.integers(-127, 128, (40, k), dtype=np.int8)
        pw = hip.PackedWeight.pack(w, sw, b)
        g = oracle.linear(x, w, 0.02, sw, b, oracle.KIND_F32_GELU)
        so = float(oracle.calibrate_out_scale(g)) or 1.0
        xd = torch.from_numpy(np.ascontiguousarray(hip.to_t16x32(x, fill=11))).cuda()
        say(f"split limits k={k}")
        for kind in (0, 4):
            y = pw.run(xd, 0.02, kind, out_scale=so, x_layout=1, y_layout=1 if kind == 4 else 0, m_tokens=40)
            torch.cuda.synchronize()
            path = hip.last_path()
            assert path.startswith("split") == want_split, path
            if want_split:
                assert "kw=16 wpw=2" in path, path
            got = y.cpu().numpy()
            if kind == 4:
                got = hip.from_t16x32(got, 40, 96)
            check(kind, got, oracle.linear(x, w, 0.02, sw, b, kind, so=so), f"k={k} kind={kind} {path}")
        pw.free()


@pytest.mark.parametrize("n", [0, 1, 15, 16, 17, 1000, 4096 * 768 + 5])
def test_quantize_act(hip, n):
    import torch
    rng = np.random.default_rng(n)
    x = (rng.standard_normal(n) * 3.0).astype(np.float32)
    if n > 20:
        x[:8] = np.array([0.5, 1.5, 2.5, -0.5, -2.5, 1e6, -1e6, 126.5], np.float32) * np.float32(0.02)
    ref = oracle.quantize(x, 0.02)
    xd = torch.from_numpy(x).cuda()
    q = hip.quantize_act(xd, 0.02)
    torch.cuda.synchronize()
    assert np.array_equal(q.cpu().numpy(), ref)
    if n > 20:  # offset view: scalar path
        q2 = hip.quantize_act(xd[1:].contiguous()[0:n - 1], 0.02)
        big = torch.zeros(n + 4, dtype=torch.float32, device="cuda")
        big[1:n + 1] = xd
        q3 = torch.zeros(n + 4, dtype=torch.int8, device="cuda")
        hip.quantize_act(big[1:n + 1], 0.02, out=q3[2:n + 2])
        torch.cuda.synchronize()
        assert np.array_equal(q2.cpu().numpy(), ref[1:])
        assert np.array_equal(q3[2:n + 2].cpu().numpy(), ref)


# ---------------------------------------------------------------------------
# workloads at their real sizes

def _gpu_chain_vs_oracle(hip, wl, calib):
    """Every op on the GPU with the oracle's own input for that op, full batch."""
    outs, scales, ins = ochain.run(wl, calib=calib)
    for layer, op in wk.op_list(wl):
        key = ochain.op_key(layer, op.name)
        wd = wk.op_weight(wl, layer, op)
        x, sx = ins[key]
        kind = KINDS[wl.op_kind(layer, op)]
        so = float(calib.get(key, 1.0))
        say(f"{wl.name} {key} kind={kind} m={x.shape[0]} n={op.n_out} k={op.k_in}")
        pw = hip.PackedWeight.pack(wd["w"], wd["sw"], wd["b"])
        got = run_gpu(hip, pw, x, sx, kind, so)
        check(kind, got, outs[key], f"{wl.name} {key}")
        acc_gpu = run_gpu(hip, pw, x, sx, 0)
        assert np.array_equal(acc_gpu, oracle.acc(x, wd["w"])), f"{wl.name} {key}: int32"
        pw.free()


@pytest.mark.parametrize("name", ["c0", "c1", "c2"])
def test_workload_full(hip, name):
    wl = wk.workloads()[name]
    _gpu_chain_vs_oracle(hip, wl, _calib()[name])


@pytest.mark.parametrize("name", [n for n in wk.workloads() if n.startswith("c3_")])
def test_workload_latency_stack(hip, name):
    wl = wk.workloads()[name]
    _gpu_chain_vs_oracle(hip, wl, _calib()[name])


@pytest.mark.parametrize("name", ["c4", "c4_bertl"])
def test_workload_full_size_sampled(hip, name):
    """M = 49152: GPU runs the whole batch; the oracle checks sampled rows."""
    import torch
    wl = wk.workloads()[name]
    calib = _calib()[name]
    rng = np.random.default_rng(123)
    rows = np.unique(np.concatenate([[0, 1, wl.m - 1, wl.m - 64, wl.m // 2],
                                     rng.choice(wl.m, 250, replace=False)]))
    for layer, op in wk.op_list(wl):
        key = ochain.op_key(layer, op.name)
        src = wl.op_src(layer, op)
        sx = float(wk.SX) if src == "seeded" else float(calib[src])
        kind = KINDS[wl.op_kind(layer, op)]
        so = float(calib.get(key, 1.0))
        x = wk.op_seeded_x(wl, layer, op)
        wd = wk.op_weight(wl, layer, op)
        say(f"{name} {key} kind={kind} m={wl.m} n={op.n_out} k={op.k_in} (sampled rows)")
        pw = hip.PackedWeight.pack(wd["w"], wd["sw"], wd["b"])
        xd = torch.from_numpy(x).cuda()
        for kd in (kind, 0):
            y = pw.run(xd, sx, kd, out_scale=so)
            torch.cuda.synchronize()
            got = y[torch.from_numpy(rows).cuda()].cpu().numpy()
            ref = oracle.linear(x[rows], wd["w"], sx, wd["sw"], wd["b"], kd, so=so)
            check(kd, got, ref, f"{name} {key} kind {kd}")
            del y
        pw.free()
        del xd


@pytest.mark.parametrize("so", [0.2, 0.05, 0.02, 0.015, 0.012, 0.01, 3.0, 40.0])
def test_gelu_requant_across_output_scales(hip, so):
    """The int8 GELU epilogue over output scales that exercise the step table
    (including codes of -1 in GELU's negative dip, so <= 0.34; the table
    spans only where codes change, so it serves scales down to 0.015) and the
    erf path the library falls back to below that, when a table cell would
    hold two changes."""
    rng = np.random.default_rng(int(so * 1000))
    w = wk.random_block_sparse(256, 768, 0.15, rng)
    sw = rng.uniform(0.001, 0.01, 256).astype(np.float32)
    b = rng.normal(0, 0.5, 256).astype(np.float32)
    x = rng.integers(-127, 128, (300, 768), dtype=np.int8)
    pw = hip.PackedWeight.pack(w, sw, b)
    say(f"gelu requant so={so}")
    got = run_gpu(hip, pw, x, 0.02, 4, so)
    path = hip.last_path()
    ref = oracle.linear(x, w, 0.02, sw, b, 4, so=so)
    check(4, got, ref, f"i8_gelu so={so} [{path}]")
    # the library takes erf exactly when the scale admits no step table
    no_table = hip.gelu_table_codes(so, np.zeros(1, np.float32)) is None
    assert no_table == (so < 0.015), so
    assert path.endswith(" gelu=erf") == no_table, path
    if so <= 0.34:
        assert (ref == -1).any() or so > 0.3  # the dip reaches code -1
