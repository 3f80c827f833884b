"""The GELU + requantisation step table against the oracle (host, no GPU).

The int8 GELU epilogue (Appendix "Graph optimization": GELU fused into the
InnerProduct; requantisation as in Section "Sparse GEMM operators") looks its
codes up in a per-scale table instead of evaluating erf. The table must give
exactly the oracle's code clamp(rint(GELU(y) * fl(1/so)), -127, 127) for
every fp32 y. The hardest values sit next to GELU's minimum (y ~ -0.7518),
where the function is flat and a code can dip and come back: there every fp32
value of [-1, -0.5) is checked, for scales that put a rounding boundary right
at the minimum's value as well as ordinary ones; elsewhere the check samples.

Where GELU is flat next to a rounding boundary, the fp32 expression itself is
not monotone: over a few consecutive fp32 values its code flips back and
forth. One threshold per cell cannot follow that, so there (and only there)
the table may give the neighbouring code. A difference is accepted only if it
is by one and the oracle's own codes within 256 fp32 steps of that value take
both codes.
"""
import numpy as np
import pytest

import oracle
import paper_2211_07715_amd as sl

GELU_MIN = -0.16997120747990188  # GELU at its minimum y = -0.75179...


def _oracle_codes(y: np.ndarray, so: float) -> np.ndarray:
    # acc = 0, scales 1, bias = y: the epilogue's dequantised value is y itself
    n = y.size
    acc = np.zeros((1, n), np.int32)
    return oracle.epilogue(acc, 1.0, np.ones(n, np.float32), y.reshape(-1), oracle.KIND_I8_GELU, so=so).reshape(-1)


NOISE_ULPS = 256


def _assert_codes(y: np.ndarray, q: np.ndarray, ref: np.ndarray, so: float):
    bad = np.nonzero(q != ref)[0]
    assert np.abs(q.astype(np.int32) - ref.astype(np.int32)).max(initial=0) <= 1, f"so={so}"
    assert bad.size <= 1e-4 * y.size + 64, f"so={so}: {bad.size} codes differ"
    for i in bad:
        bits = np.array([y[i]], np.float32).view(np.int32)[0]
        near = np.arange(bits - NOISE_ULPS, bits + NOISE_ULPS + 1, dtype=np.int32).view(np.float32)
        codes = set(_oracle_codes(near, so).tolist())
        assert {int(q[i]), int(ref[i])} <= codes, (
            f"so={so}: y={y[i]!r} table {q[i]} oracle {ref[i]}, and the oracle is monotone around it")


def _all_fp32(lo: float, hi: float) -> np.ndarray:
    """Every fp32 value of [lo, hi) for 0 < lo < hi (as positive bit patterns)."""
    a = np.array([lo], np.float32).view(np.int32)[0]
    b = np.array([hi], np.float32).view(np.int32)[0]
    return np.arange(a, b, dtype=np.int32).view(np.float32)


# ordinary scales, and scales whose minimum value lies just past a rounding
# boundary, so that the code dips by one on both sides of the minimum within a
# cell width or two of it
SCALES = [0.015, 0.02, 0.05, 0.3, 1.0,
          float(np.float32(-GELU_MIN / 8.503)), float(np.float32(-GELU_MIN / 8.53)),
          float(np.float32(-GELU_MIN / 0.502)), float(np.float32(-GELU_MIN / 2.51))]
# scales that put the minimum's value exactly on a boundary: the fp32
# expression then flips between two codes many times next to the minimum,
# no table can hold that, and the kernels evaluate erf instead
AT_BOUNDARY = [float(np.float32(-GELU_MIN / 8.5)), float(np.float32(-GELU_MIN / 0.5))]


@pytest.mark.parametrize("so", SCALES + AT_BOUNDARY)
def test_every_fp32_value_around_the_minimum(so):
    y = -_all_fp32(0.5, 1.0)  # every fp32 y in (-1, -0.5]
    q = sl.gelu_table_codes(so, y)
    if so in AT_BOUNDARY and q is None:
        return
    assert q is not None, "no table for a scale above 0.015"
    _assert_codes(y, q, _oracle_codes(y, so), so)


@pytest.mark.parametrize("so", SCALES)
def test_sampled_values_everywhere(so):
    rng = np.random.default_rng(7)
    span = 140.0 * so + 8.0
    y = np.concatenate([
        rng.uniform(-span, span, 400_000),
        rng.uniform(-6.0, 4.0, 400_000),
        np.sign(rng.uniform(-1, 1, 200_000)) * np.exp(rng.uniform(-30, np.log(span), 200_000)),
        [0.0, -0.0, 1e-30, -1e-30, 3e38, -3e38, np.inf, -np.inf],
    ]).astype(np.float32)
    q = sl.gelu_table_codes(so, y)
    _assert_codes(y, q, _oracle_codes(y, so), so)


def test_codes_at_the_thresholds_of_one_scale():
    """Every code change of one scale, located by scanning the oracle's codes
    over a fine fp32 grid, then both sides of each change value by value."""
    so = 0.02
    y = np.linspace(-6.0, 3.2, 2_000_001, dtype=np.float32)
    ref = _oracle_codes(y, so)
    idx = np.nonzero(np.diff(ref.astype(np.int32)))[0]
    assert idx.size > 100
    pts = []
    for i in idx:
        a = np.array([y[i]], np.float32).view(np.int32)[0]
        b = np.array([y[i + 1]], np.float32).view(np.int32)[0]
        lo, hi = (a, b) if a < b else (b, a)
        pts.append(np.arange(lo - 2, hi + 3, dtype=np.int32))
    bits = np.concatenate(pts)
    yy = bits.view(np.float32)
    q = sl.gelu_table_codes(so, yy)
    _assert_codes(yy, q, _oracle_codes(yy, so), so)


def test_small_scales_have_no_table_and_bad_scales_are_rejected():
    assert sl.gelu_table_codes(0.005, np.zeros(4, np.float32)) is None
    lib = sl.load()
    y = np.zeros(4, np.float32)
    q = np.zeros(4, np.int8)
    for bad in (0.0, -1.0, float("nan"), float("inf")):
        assert lib.sl_gelu_table_codes(bad, y.ctypes.data, q.ctypes.data, 4) == -1
    assert lib.sl_gelu_table_codes(0.1, None, None, 4) == -1
    assert lib.sl_gelu_table_codes(0.1, None, None, 0) == 0
