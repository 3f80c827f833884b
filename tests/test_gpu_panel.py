"""GPU parity of the weight-stationary kernel (the whole channel-group panel
resident in LDS) against the CPU oracle, through the C ABI.

Every compiled workgroup shape runs every epilogue kind on shapes with ragged
token, channel and column tails, in each activation layout pairing, and the
kernel that actually ran is checked by name (sl_last_path). Bars as in
test_gpu_parity.py: int32 bit-exact, fp32 max|err| <= 1e-5 * max|ref|, int8
within 1 LSB in at most 0.01 % of the elements.
"""
import numpy as np
import pytest

import oracle
from test_gpu_parity import KINDS, _case, check, say

pytestmark = pytest.mark.gpu

T = 1  # SL_LAYOUT_T16X32
SHAPES = ["6,2,12,2", "6,2,8,2", "4,2,8,2", "2,2,8,4", "2,4,4,2"]

# (m, n, k, density): k a multiple of 16 so that row-major rows qualify too
CASES = [
    (1, 4, 16, 0.35),
    (33, 100, 272, 0.35),      # ragged channel tile and last window
    (20, 32, 256, 0.0),        # nothing stored: bias only
    (50, 48, 768, 1.0),        # every window of every tile overflows
    (130, 200, 1024, 0.1),
    (300, 96, 768, 0.3),
    (65, 768, 3072, 0.1),      # DistilBERT FFN2 shape
    (257, 3072, 768, 0.1),     # DistilBERT FFN1 shape
    (40, 64, 4096, 0.2),
]


def _refs(x, w, sw, b):
    out = {}
    for name, kind in KINDS.items():
        so = 1.0
        if kind in (3, 4):
            g = oracle.linear(x, w, 0.02, sw, b, 1 if kind == 3 else 2)
            so = float(oracle.calibrate_out_scale(g)) or 1.0
        out[kind] = (so, oracle.linear(x, w, 0.02, sw, b, kind, so=so))
    return out


@pytest.mark.parametrize("m,n,k,density", CASES)
def test_panel_every_shape_kind_layout(hip, monkeypatch, m, n, k, density):
    import torch
    w, sw, b, rng = _case(n, k, density, 7 * m + 3 * n + k + int(100 * density))
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    refs = _refs(x, w, sw, b)
    pw = hip.PackedWeight.pack(w, sw, b)
    x_rows = torch.from_numpy(x).cuda()
    x_blk = torch.from_numpy(np.ascontiguousarray(hip.to_t16x32(x, fill=77))).cuda()
    monkeypatch.setenv("SL_PATH", "panel")
    ran = 0
    for shape in SHAPES:
        monkeypatch.setenv("SL_PTILE", shape)
        for xl, yl in [(0, 0), (T, 0), (T, T), (0, T)]:
            for name, kind in KINDS.items():
                if yl == T and kind not in (3, 4):
                    continue
                so, ref = refs[kind]
                say(f"panel {shape} m={m} n={n} k={k} d={density} layouts=({xl},{yl}) {name}")
                y = pw.run(x_blk if xl == T else x_rows, 0.02, kind, out_scale=so, x_layout=xl, y_layout=yl,
                           m_tokens=m)
                torch.cuda.synchronize()
                path = hip.last_path()
                got = y.cpu().numpy()
                if yl == T:
                    got = hip.from_t16x32(got, m, n)
                check(kind, got, ref, f"{path} {name} m={m} n={n} k={k} layouts=({xl},{yl})")
                if path.startswith(f"panel {shape} "):
                    ran += 1
    pw.free()
    # the panel fits for every case but the densest large ones
    assert ran > 0, "the weight-stationary kernel never ran"


def test_panel_runs_at_distilbert_ffn_shapes(hip, monkeypatch):
    """The chooser takes the weight-stationary kernel for both FFN GEMMs at
    90 % and 80 % sparsity (4096 tokens), and their outputs match the oracle
    on sampled rows."""
    import torch
    import workloads as wk
    monkeypatch.setenv("SL_PATH", "panel")
    m = 4096
    for (n, k) in [(3072, 768), (768, 3072)]:
        for sparsity in (0.9, 0.8):
            wd = wk.make_weight(n, k, sparsity, seed=5)
            x = wk.make_x(m, k, seed=5)
            pw = hip.PackedWeight.pack(wd["w"], wd["sw"], wd["b"])
            y = pw.run(torch.from_numpy(x).cuda(), 0.02, KINDS["acc_i32"])
            torch.cuda.synchronize()
            path = hip.last_path()
            say(f"ffn {n}x{k} s={sparsity}: {path}")
            assert path.startswith("panel"), path
            rows = np.random.default_rng(0).choice(m, 64, replace=False)
            rows.sort()
            ref = oracle.acc(np.ascontiguousarray(x[rows]), wd["w"])
            check(0, y.cpu().numpy()[rows], ref, f"{n}x{k} s={sparsity}")
            pw.free()


def test_default_path_choice(hip, monkeypatch):
    """Without SL_PATH few tokens (at most 1280 work items of 16 tokens x 32
    channels) go to the split-reduction kernel; beyond that the
    weight-stationary kernel runs for short reductions (K <= 1024) of
    widening layers (DistilBERT QKV and FFN1), of long token slices, or
    unless the direct kernel's work items make one round of the CUs that
    keeps most of them busy (not so for the square 768 layer at 1024 or
    8192 tokens, or 1024x1024 at 4096); the direct kernel elsewhere: FFN2
    (K = 3072) and the square attention-output layer at 2048 and 4096
    tokens."""
    import torch
    import workloads as wk
    monkeypatch.delenv("SL_PATH", raising=False)
    monkeypatch.delenv("SL_PTILE", raising=False)
    for (n, k, m, s, want) in [(3072, 768, 4096, 0.9, "panel 6,2,12,2"), (3072, 768, 4096, 0.8, "panel 6,2,12,2"),
                               (3072, 768, 16384, 0.8, "panel 6,2,12,2"), (2304, 768, 4096, 0.8, "panel 6,2,12,2"),
                               (2304, 768, 384, 0.8, "panel"),
                               (768, 3072, 4096, 0.9, "direct"), (768, 768, 4096, 0.8, "direct"),
                               (768, 768, 128, 0.9, "split"), (3072, 768, 128, 0.8, "split"),
                               (768, 3072, 384, 0.8, "split"), (768, 768, 1024, 0.8, "panel"),
                               (768, 768, 2048, 0.8, "direct"), (1024, 1024, 4096, 0.8, "panel"),
                               (768, 768, 8192, 0.8, "panel")]:
        wd = wk.make_weight(n, k, s, seed=3)
        x = wk.make_x(m, k, seed=3)
        pw = hip.PackedWeight.pack(wd["w"], wd["sw"], wd["b"])
        xb = torch.from_numpy(np.ascontiguousarray(hip.to_t16x32(x))).cuda()
        y = pw.run(xb, 0.02, KINDS["acc_i32"], x_layout=T, m_tokens=m)
        torch.cuda.synchronize()
        path = hip.last_path()
        say(f"default {n}x{k} s={s} m={m}: {path}")
        assert path.startswith(want), path
        rows = np.arange(0, m, max(1, m // 48))
        check(0, y.cpu().numpy()[rows], oracle.acc(np.ascontiguousarray(x[rows]), wd["w"]), f"{n}x{k} m={m}")
        pw.free()


def test_panel_falls_back_when_no_panel_fits(hip, monkeypatch):
    """A reduction too long for any channel group's panel to fit in LDS
    (k = 16384: 128 windows, over 270 KB for two tiles) gets no panel image;
    SL_PATH=panel then runs another kernel, with the same results."""
    import torch
    m, n, k = 20, 8, 16384
    w, sw, b, rng = _case(n, k, 0.3, 11)
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    pw = hip.PackedWeight.pack(w, sw, b)
    monkeypatch.setenv("SL_PATH", "panel")
    monkeypatch.delenv("SL_PTILE", raising=False)
    for xl in (0, T):
        xd = torch.from_numpy(np.ascontiguousarray(hip.to_t16x32(x, fill=5) if xl == T else x)).cuda()
        for name in ("acc_i32", "f32"):
            kind = KINDS[name]
            say(f"no panel fits: k={k} layout={xl} {name}")
            y = pw.run(xd, 0.02, kind, x_layout=xl, m_tokens=m)
            torch.cuda.synchronize()
            path = hip.last_path()
            assert not path.startswith("panel"), path
            check(kind, y.cpu().numpy(), oracle.linear(x, w, 0.02, sw, b, kind), f"{path} {name} layout={xl}")
    pw.free()
