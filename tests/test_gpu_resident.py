"""GPU parity of the register-resident kernel against the CPU oracle, through
the C ABI.

The kernel keeps each wave's main weight operands in registers, streams token
passes through LDS, and folds the rare third and fourth blocks of an aligned
4-column group into consolidated overflow operands whose dense operand is
gathered 4 bytes a slot; K beyond one wave's 768-column slice is split over
2 or 4 waves and summed exactly through LDS. Every epilogue kind runs in every
activation layout pairing on shapes with ragged token, channel and column
tails, empty and fully dense weights (every group overflows), and each split
of the reduction; sl_last_path() confirms the kernel that ran. Bars as in
test_gpu_parity.py: int32 bit-exact, fp32 max|err| <= 1e-5 * max|ref|, int8
within 1 LSB in at most 0.01 % of the elements.
"""
import numpy as np
import pytest

import oracle
from test_gpu_parity import KINDS, _case, check, say

pytestmark = pytest.mark.gpu

T = 1  # SL_LAYOUT_T16X32

# (m, n, k, density); k a multiple of 16 so that row-major rows qualify too
CASES = [
    (1, 4, 16, 0.35),
    (33, 100, 272, 0.35),      # ragged channel tile and last window
    (20, 32, 256, 0.0),        # nothing stored: bias only
    (50, 48, 768, 1.0),        # every group of every block-row holds 4 blocks
    (130, 200, 1024, 0.1),     # reduction split over 2 waves
    (300, 400, 768, 0.3),      # several channel groups and token slices
    (65, 768, 3072, 0.1),      # DistilBERT FFN2 shape: split over 4 waves
    (257, 3072, 768, 0.1),     # DistilBERT FFN1 shape
    (40, 64, 2000, 0.5),       # ragged split reduction, many overflows
    (17, 96, 3072, 0.2),       # split over 4 waves, an overflow operand per tile and slice
    (17, 96, 3072, 1.0),       # dense: the overflow operands exceed LDS, another kernel runs
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
def test_resident_every_kind_and_layout(hip, monkeypatch, m, n, k, density):
    import torch
    w, sw, b, rng = _case(n, k, density, 11 * m + 5 * n + k + int(100 * density))
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    refs = _refs(x, w, sw, b)
    pw = hip.PackedWeight.pack(w, sw, b)
    x_rows = torch.from_numpy(x).cuda()
    x_blk = torch.from_numpy(np.ascontiguousarray(hip.to_t16x32(x, fill=77))).cuda()
    monkeypatch.setenv("SL_PATH", "resident")
    for xl, yl in [(0, 0), (T, 0), (T, T), (0, T)]:
        for name, kind in KINDS.items():
            if yl == T and kind not in (3, 4):
                continue
            so, ref = refs[kind]
            say(f"resident m={m} n={n} k={k} d={density} layouts=({xl},{yl}) {name}")
            y = pw.run(x_blk if xl == T else x_rows, 0.02, kind, out_scale=so, x_layout=xl, y_layout=yl,
                       m_tokens=m)
            torch.cuda.synchronize()
            path = hip.last_path()
            if not (k == 3072 and density == 1.0):
                assert path.startswith("resident "), path
            got = y.cpu().numpy()
            if yl == T:
                got = hip.from_t16x32(got, m, n)
            check(kind, got, ref, f"{path} {name} m={m} n={n} k={k} layouts=({xl},{yl})")
    pw.free()
