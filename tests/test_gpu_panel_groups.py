"""GPU parity of the weight-stationary kernel when each wave walks several
token groups (one token slice per channel group, SL_PSLICES=1), through the
C ABI: the operand ring reading ahead into the next group's first window,
the ring-slot move after an odd window count (2-tile groups), the token rows
of the next group loading during an epilogue, and the int8 epilogues' table
reads across groups. Every compiled shape, window counts 1, 3, 6 and 8,
every epilogue kind, row-major and block-layout activations; a ragged last
token group. Bars as in test_gpu_parity.py.
"""
import numpy as np
import pytest

import oracle
from test_gpu_panel import SHAPES, T, _refs
from test_gpu_parity import KINDS, _case, check, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("k", [128, 384, 768, 1024])
def test_panel_many_groups_per_wave(hip, monkeypatch, k):
    import torch
    n = 96
    w, sw, b, rng = _case(n, k, 0.15, 31 + k)
    monkeypatch.setenv("SL_PATH", "panel")
    monkeypatch.setenv("SL_PSLICES", "1")
    pw = hip.PackedWeight.pack(w, sw, b)
    ran = 0
    for shape in SHAPES:
        nt, st, nwv, r = (int(v) for v in shape.split(","))
        # at least 2 token groups a wave and a ragged last group
        m = 16 * st * nwv * 2 + 16 * st + 5
        x = rng.integers(-127, 128, (m, k), dtype=np.int8)
        refs = _refs(x, w, sw, b)
        monkeypatch.setenv("SL_PTILE", shape)
        x_rows = torch.from_numpy(x).cuda()
        x_blk = torch.from_numpy(np.ascontiguousarray(hip.to_t16x32(x, fill=9))).cuda()
        for xl, yl in [(0, 0), (T, T)]:
            for name, kind in KINDS.items():
                so, ref = refs[kind]
                yl_k = yl if kind in (3, 4) else 0
                say(f"panel groups {shape} m={m} k={k} layouts=({xl},{yl_k}) {name}")
                y = pw.run(x_blk if xl == T else x_rows, 0.02, kind, out_scale=so, x_layout=xl, y_layout=yl_k,
                           m_tokens=m)
                torch.cuda.synchronize()
                path = hip.last_path()
                assert path.startswith(f"panel {shape}") and "slices=1x" in path, path
                got = y.cpu().numpy()
                if yl_k == T:
                    got = hip.from_t16x32(got, m, n)
                check(kind, got, ref, f"{path} {name} m={m} k={k} layouts=({xl},{yl_k})")
                ran += 1
    pw.free()
    assert ran == len(SHAPES) * 2 * len(KINDS)
