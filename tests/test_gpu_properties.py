"""GPU property test (hypothesis, derandomised): over generated shapes, masks,
kernels and activation layouts, the int32 accumulators of the HIP path are
bit-identical to the oracle's, and the fp32 outputs meet the fp32 bar.

Shapes span several tiles with ragged token, channel and column tails; k is
a multiple of 16 so that every kernel (staged, direct, weight-stationary, split)
accepts row-major rows. The kernel that ran is recorded in the failure text.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from test_gpu_parity import check

pytestmark = pytest.mark.gpu

PATHS = [{}, {"SL_PATH": "staged"}, {"SL_PATH": "direct"}, {"SL_PATH": "panel"}, {"SL_PATH": "split"}]


@settings(max_examples=40, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])
@given(m=st.integers(1, 90), n4=st.integers(1, 48), k16=st.integers(1, 48),
       density=st.sampled_from([0.0, 0.05, 0.2, 0.5, 1.0]), path=st.integers(0, len(PATHS) - 1),
       block_x=st.booleans(), seed=st.integers(0, 2 ** 31 - 1))
def test_gpu_int32_and_fp32_match_oracle(hip, monkeypatch, m, n4, k16, density, path, block_x, seed):
    import torch
    n, k = 4 * n4, 16 * k16
    rng = np.random.default_rng(seed)
    keep = rng.random((n // 4, k)) < density
    w = (rng.integers(-127, 128, (n, k), dtype=np.int8) * np.repeat(keep, 4, axis=0).astype(np.int8)).astype(np.int8)
    sw = rng.uniform(0.001, 0.01, n).astype(np.float32)
    b = rng.normal(0, 0.02, n).astype(np.float32)
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    for key in ("SL_PATH", "SL_PTILE", "SL_DTILE", "SL_TILE"):
        monkeypatch.delenv(key, raising=False)
    for key, val in PATHS[path].items():
        monkeypatch.setenv(key, val)
    pw = hip.PackedWeight.pack(w, sw, b)
    try:
        if block_x:
            xd = torch.from_numpy(np.ascontiguousarray(hip.to_t16x32(x, fill=-3))).cuda()
        else:
            xd = torch.from_numpy(x).cuda()
        lay = 1 if block_x else 0
        acc = pw.run(xd, 0.02, 0, x_layout=lay, m_tokens=m)
        torch.cuda.synchronize()
        what = f"m={m} n={n} k={k} d={density} {PATHS[path]} block_x={block_x}: {hip.last_path()}"
        check(0, acc.cpu().numpy(), oracle.acc(x, w), what)
        y = pw.run(xd, 0.02, 1, x_layout=lay, m_tokens=m)
        torch.cuda.synchronize()
        check(1, y.cpu().numpy(), oracle.linear(x, w, 0.02, sw, b, oracle.KIND_F32), what)
    finally:
        pw.free()
