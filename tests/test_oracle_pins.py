"""Pins for the CPU oracle (CPU only).

The oracle is the plain definition of the layer (dense int32 contraction, then
a fixed-order fp32 epilogue). These tests tie it to things other than itself:
brute-force integer sums in pure Python, numpy's int64 matmul, algebraic
invariants of the block-sparse product, the exact (fp64) values of the
epilogue formulas within their rounding bounds, closed-form special cases of
GELU and of round-half-to-even requantisation, and a hand-worked example.
A plausible slip in the oracle (a transposed operand, a wrong scale index, a
dropped bias, a wrong GELU constant, truncating instead of rounding, a
-128 clamp) fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from workloads import random_block_sparse, make_weight, block_keep_mask

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
U = 2.0 ** -24  # unit roundoff of fp32


def brute_acc(x, w):
    """Pure-Python integer sums, one element at a time."""
    m, k = x.shape
    n = w.shape[0]
    out = [[0] * n for _ in range(m)]
    for i in range(m):
        for j in range(n):
            s = 0
            for t in range(k):
                s += int(x[i, t]) * int(w[j, t])
            out[i][j] = s
    return np.array(out, dtype=np.int64)


@pytest.mark.parametrize("m,n,k", [(1, 4, 1), (2, 4, 2), (3, 8, 7), (5, 12, 33), (16, 8, 64), (7, 20, 5)])
def test_acc_brute_force(m, n, k):
    rng = np.random.default_rng(1000 + m * 100 + n * 10 + k)
    for density in (0.0, 0.3, 1.0):
        x = rng.integers(-127, 128, (m, k), dtype=np.int8)
        w = random_block_sparse(n, k, density, rng)
        assert np.array_equal(oracle.acc(x, w).astype(np.int64), brute_acc(x, w))


def test_acc_extreme_values_brute_force():
    # all-(-127) / all-127 operands: the largest magnitudes the int8 range allows
    x = np.full((2, 9), -127, dtype=np.int8)
    x[1] = 127
    w = np.full((4, 9), 127, dtype=np.int8)
    w[2] = -127
    assert np.array_equal(oracle.acc(x, w).astype(np.int64), brute_acc(x, w))
    assert oracle.acc(x, w)[0, 0] == -127 * 127 * 9


def test_acc_numpy_int64_large():
    rng = np.random.default_rng(7)
    for (m, n, k) in [(64, 3072, 768), (33, 768, 3072), (5, 1024, 4096)]:
        x = rng.integers(-127, 128, (m, k), dtype=np.int8)
        w = random_block_sparse(n, k, 0.15, rng)
        ref = x.astype(np.int64) @ w.astype(np.int64).T
        assert np.array_equal(oracle.acc(x, w).astype(np.int64), ref)


def test_acc_worst_case_no_overflow():
    # |acc| = 127*127*4096 = 66,064,384 < 2^31: exact at the largest K used
    x = np.full((1, 4096), 127, dtype=np.int8)
    w = np.full((4, 4096), -127, dtype=np.int8)
    assert int(oracle.acc(x, w)[0, 0]) == -127 * 127 * 4096


def test_invariant_zero_blocks_contribute_nothing():
    rng = np.random.default_rng(11)
    n, k, m = 16, 50, 9
    w = random_block_sparse(n, k, 0.3, rng)
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    base = oracle.acc(x, w)
    for g in range(n // 4):
        support = np.any(w[4 * g:4 * g + 4] != 0, axis=0)
        x2 = x.copy()
        x2[:, ~support] = rng.integers(-127, 128, (m, int((~support).sum())), dtype=np.int8)
        out = oracle.acc(x2, w)
        assert np.array_equal(out[:, 4 * g:4 * g + 4], base[:, 4 * g:4 * g + 4])


def test_invariant_all_zero_weight_gives_bias():
    rng = np.random.default_rng(12)
    m, n, k = 6, 12, 40
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    w = np.zeros((n, k), dtype=np.int8)
    sw = rng.uniform(0.001, 0.01, n).astype(np.float32)
    b = rng.normal(0, 0.02, n).astype(np.float32)
    assert not oracle.acc(x, w).any()
    y = oracle.linear(x, w, 0.02, sw, b, oracle.KIND_F32)
    assert np.array_equal(y, np.broadcast_to(b, (m, n)))
    y0 = oracle.linear(x, w, 0.02, sw, None, oracle.KIND_F32)
    assert not y0.any()


def test_invariant_identity_reproduces_input():
    rng = np.random.default_rng(13)
    k = 64
    x = rng.integers(-127, 128, (10, k), dtype=np.int8)
    w = np.eye(k, dtype=np.int8)  # 4 stored blocks per block-row, 1 on the diagonal
    assert np.array_equal(oracle.acc(x, w), x.astype(np.int32))
    y = oracle.linear(x, w, 1.0, np.ones(k, np.float32), None, oracle.KIND_F32)
    assert np.array_equal(y, x.astype(np.float32))
    q = oracle.linear(x, w, 1.0, np.ones(k, np.float32), None, oracle.KIND_I8, so=1.0)
    assert np.array_equal(q, x)


def test_invariant_linearity_and_column_permutation():
    rng = np.random.default_rng(14)
    m, n, k = 7, 16, 30
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    w1 = random_block_sparse(n, k, 0.4, rng) // 2
    w2 = random_block_sparse(n, k, 0.4, rng) // 2
    a12 = oracle.acc(x, (w1 + w2).astype(np.int8))
    assert np.array_equal(a12, oracle.acc(x, w1) + oracle.acc(x, w2))
    perm = rng.permutation(k)
    assert np.array_equal(oracle.acc(x[:, perm], w1[:, perm]), oracle.acc(x, w1))


def test_invariant_row_subsets_are_independent():
    rng = np.random.default_rng(15)
    x = rng.integers(-127, 128, (40, 32), dtype=np.int8)
    w = random_block_sparse(8, 32, 0.5, rng)
    sw = rng.uniform(0.001, 0.01, 8).astype(np.float32)
    full = oracle.linear(x, w, 0.02, sw, None, oracle.KIND_F32_GELU)
    idx = np.array([39, 0, 17, 17, 3])
    assert np.array_equal(oracle.linear(x[idx], w, 0.02, sw, None, oracle.KIND_F32_GELU), full[idx])


def _exact_y(acc, sx, sw, b):
    return acc.astype(np.float64) * (np.float64(sx) * sw.astype(np.float64))[None, :] + b.astype(np.float64)[None, :]


def test_dequant_within_rounding_bound_of_exact():
    """fp32 y vs exact y: three roundings (s, acc*s, +b) bound the error."""
    rng = np.random.default_rng(16)
    m, n, k = 64, 32, 3072
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    w = random_block_sparse(n, k, 0.2, rng)
    sw = rng.uniform(0.001, 0.01, n).astype(np.float32)
    b = rng.normal(0, 0.02, n).astype(np.float32)
    sx = np.float32(0.02)
    a = oracle.acc(x, w)
    y = oracle.linear(x, w, sx, sw, b, oracle.KIND_F32).astype(np.float64)
    ex = _exact_y(a, sx, sw, b)
    prod = np.abs(a.astype(np.float64) * (np.float64(sx) * sw)[None, :])
    bound = prod * 3.01 * U + np.abs(ex) * 1.01 * U
    assert np.all(np.abs(y - ex) <= bound)
    # a dropped bias or a wrong scale index would blow far past the bound
    assert np.abs(y - ex).max() < 1e-5 * np.abs(ex).max()


def test_gelu_special_cases_and_exact_values():
    ys = np.concatenate([np.linspace(-8, 8, 4001), [0.0, 1e-30, -1e-30, 1e-3, -1e-3, 30.0, -30.0]]).astype(np.float32)
    g = oracle.gelu(ys).astype(np.float64)
    ex = np.array([0.5 * v * (1.0 + math.erf(v / math.sqrt(2.0))) for v in ys.astype(np.float64)])
    # erf form, not the tanh approximation (which is off by up to ~5e-4 near |y|=2)
    assert np.all(np.abs(g - ex) <= 6 * U * np.maximum(np.abs(ys), 1e-30) + 1e-37)
    assert oracle.gelu(np.array([0.0], np.float32))[0] == 0.0
    # GELU(y) - GELU(-y) = y (erf is odd)
    pos = ys[ys > 0]
    d = oracle.gelu(pos).astype(np.float64) - oracle.gelu(-pos).astype(np.float64)
    assert np.all(np.abs(d - pos) <= 4 * U * pos)
    # far tails: erf rounds to +-1 in fp32, so GELU is exactly y, resp. zero
    big = np.array([6.0, 7.5, 40.0, 1000.0], np.float32)
    assert np.array_equal(oracle.gelu(big), big)
    assert np.all(oracle.gelu(-big) == 0.0)
    # the minimum of GELU: about -0.16997 at y ~ -0.7518
    assert abs(oracle.gelu(np.array([-0.7518], np.float32))[0] + 0.169971) < 1e-5


def _epi_single(accv, sx, swv, bv, kind, so):
    return oracle.epilogue(np.array([[accv]], np.int32), sx, np.array([swv], np.float32),
                           np.array([bv], np.float32), kind, so)[0, 0]


def test_requant_round_half_to_even_and_saturation():
    # y = acc * (1 * 0.5) + 0 is exact; so = 1 -> v = acc / 2
    cases = {5: 2, 7: 4, -5: -2, -7: -4, 1: 0, -1: 0, 3: 2, 9: 4, 254: 127, 255: 127, 256: 127,
             -254: -127, -255: -127, -256: -127, 253: 126, 10_000: 127, -10_000: -127}
    for a, q in cases.items():
        assert _epi_single(a, 1.0, 0.5, 0.0, oracle.KIND_I8, 1.0) == q, a
    # never -128, even far below the range
    assert _epi_single(-2**30, 1.0, 1.0, 0.0, oracle.KIND_I8, 1.0) == -127
    # so scales before rounding: v = 3 / 2 = 1.5 -> 2 ; 2.5 -> 2
    assert _epi_single(3, 1.0, 1.0, 0.0, oracle.KIND_I8, 2.0) == 2
    assert _epi_single(5, 1.0, 1.0, 0.0, oracle.KIND_I8, 2.0) == 2


def test_requant_with_gelu_tails():
    # y = 300 -> GELU = 300 exactly -> /so=4 -> 75 ; y = -300 -> 0
    assert _epi_single(600, 1.0, 0.5, 0.0, oracle.KIND_I8_GELU, 4.0) == 75
    assert _epi_single(-600, 1.0, 0.5, 0.0, oracle.KIND_I8_GELU, 4.0) == 0


def test_requant_matches_exact_rounding_on_random_data():
    rng = np.random.default_rng(17)
    m, n, k = 32, 64, 768
    x = rng.integers(-127, 128, (m, k), dtype=np.int8)
    w = random_block_sparse(n, k, 0.2, rng)
    sw = rng.uniform(0.001, 0.01, n).astype(np.float32)
    b = rng.normal(0, 0.02, n).astype(np.float32)
    so = np.float32(0.05)
    y = oracle.linear(x, w, 0.02, sw, b, oracle.KIND_F32).astype(np.float64)
    q = oracle.linear(x, w, 0.02, sw, b, oracle.KIND_I8, so=so).astype(np.int64)
    v = y / np.float64(so)
    ref = np.clip(np.round(v), -127, 127)  # numpy rounds half to even
    # exact fp64 rounding may differ only where v sits within fp32 error of a .5
    frac = np.abs(np.abs(v - np.floor(v)) - 0.5)
    agree = (q == ref) | (frac < 1e-4)
    assert agree.all()
    assert (q == ref).mean() > 0.999


def test_quantize_contract():
    s = np.float32(0.02)
    k = np.arange(-127, 128, dtype=np.int8)
    x = k.astype(np.float32) * s  # round trip of every code
    assert np.array_equal(oracle.quantize(x, s), k)
    # ties to even, saturation at +-127
    xs = np.array([0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 126.5, 127.5, 128.0, -127.5, -1e9, 1e9], np.float32)
    exp = np.array([0, 2, 2, 0, -2, -2, 126, 127, 127, -127, -127, 127], np.int8)
    assert np.array_equal(oracle.quantize(xs, 1.0), exp)
    with pytest.raises(ValueError):
        oracle.quantize(np.array([np.nan], np.float32), 1.0)


def test_calibration_uses_full_int8_range():
    rng = np.random.default_rng(18)
    x = rng.integers(-127, 128, (64, 768), dtype=np.int8)
    wd = make_weight(3072, 768, 0.9, seed=5)
    g = oracle.linear(x, wd["w"], 0.02, wd["sw"], wd["b"], oracle.KIND_F32_GELU)
    so = oracle.calibrate_out_scale(g)
    q = oracle.quantize(g, so)
    assert np.abs(q.astype(np.int32)).max() == 127
    # requantising inside the epilogue and after it are the same decision
    q2 = oracle.linear(x, wd["w"], 0.02, wd["sw"], wd["b"], oracle.KIND_I8_GELU, so=so)
    assert np.array_equal(q, q2)


def test_generator_block_structure():
    for (n, k, s) in [(768, 768, 0.8), (3072, 768, 0.9), (16, 10, 0.5)]:
        wd = make_weight(n, k, s, seed=3)
        keep = wd["keep"]
        nb = (n // 4) * k
        assert keep.sum() == nb - int(np.floor(s * nb + 0.5))
        # every zeroed block is zero in all 4 rows
        w4 = wd["w"].reshape(n // 4, 4, k)
        assert not w4[~keep[:, None, :].repeat(4, axis=1)].any()
    rng = np.random.default_rng(0)
    a = block_keep_mask(8, 8, 0.5, np.random.default_rng(1))
    b = block_keep_mask(8, 8, 0.5, np.random.default_rng(1))
    assert np.array_equal(a, b)
    del rng


def test_hand_worked_example():
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        ex = json.load(f)
    x = np.array(ex["x"], np.int8)
    w = np.array(ex["w"], np.int8)
    sw = np.array(ex["sw"], np.float32)
    b = np.array(ex["bias"], np.float32)
    assert np.array_equal(oracle.acc(x, w), np.array(ex["acc"], np.int32))
    y = oracle.linear(x, w, ex["sx"], sw, b, oracle.KIND_F32)
    assert np.array_equal(y, np.array(ex["y_f32"], np.float32))
    q = oracle.linear(x, w, ex["sx"], sw, b, oracle.KIND_I8, so=ex["so"])
    assert np.array_equal(q, np.array(ex["q_i8"], np.int8))
    qg = oracle.linear(x, w, ex["sx"], sw, b, oracle.KIND_I8_GELU, so=ex["so"])
    assert np.array_equal(qg, np.array(ex["q_i8_gelu"], np.int8))


def test_calibration_takes_the_magnitude_of_a_negative_extreme():
    # Section "Post-training quantization": the per-tensor output scale maps the
    # largest magnitude to code 127; a signed output whose extreme is negative
    # must set it (g = [-3, 1, 2] -> max|g| = 3, so = 3/127 in fp32).
    g = np.array([[-3.0, 1.0, 2.0]], np.float32)
    assert oracle.absmax(g) == np.float32(3.0)
    so = oracle.calibrate_out_scale(g)
    assert so == np.float32(3.0) / np.float32(127.0)
    # the extreme then maps to -127 exactly, the others by rounding
    assert np.array_equal(oracle.quantize(g, so), np.array([[-127, 42, 85]], np.int8))
    # a negative extreme far below every positive value
    g2 = np.array([0.5, -100.0, 99.0, 0.0], np.float32)
    assert oracle.absmax(g2) == np.float32(100.0)


def test_chain_feeds_the_calibrated_output_scale_forward(monkeypatch):
    """Hand-worked two-op chain: op b's input scale is op a's calibrated so.

    Op a: x = [127, -64] with the seeded scale 0.02 and w_scale 50, so the
    dequantisation scale fl(0.02 * 50) is exactly 1.0 and y = acc =
    [127, -64, 63, 64]; so_a = 127 / 127 = 1.0 and the int8 codes equal y.
    Op b reads those codes with x_scale = so_a = 1.0 and w_scale 0.5:
    acc_b = [127, -64, 127, 63], y_b = acc_b * 0.5 + bias = [63.5, -32, 63.75, 31.5].
    Had op b used the seeded scale 0.02 instead, y_b would be about 50x smaller.
    """
    from oracle import chain
    import workloads as wk_mod

    ops = (wk_mod.Op("a", 0, 4, 2, 0.0, "i8"), wk_mod.Op("b", 1, 4, 4, 0.0, "f32", "a"))
    wl = wk_mod.Workload("hand", 9, 0, 1, 1, ops)
    x_a = np.array([[127, -64]], np.int8)
    monkeypatch.setattr(wk_mod, "op_seeded_x", lambda *a, **k: x_a.copy())
    weights = {
        "L0.a": {"w": np.array([[1, 0], [0, 1], [1, 1], [0, -1]], np.int8),
                 "sw": np.full(4, 50.0, np.float32), "b": np.zeros(4, np.float32)},
        "L0.b": {"w": np.array([[1, 0, 0, 0], [0, 1, 0, 0], [0, 0, 1, 1], [1, 0, 0, -1]], np.int8),
                 "sw": np.full(4, 0.5, np.float32), "b": np.array([0, 0, 0.25, 0], np.float32)},
    }
    outs, scales, ins = chain.run(wl, weights=weights)
    assert scales["L0.a"] == np.float32(1.0)
    assert np.array_equal(outs["L0.a"], np.array([[127, -64, 63, 64]], np.int8))
    assert ins["L0.b"][1] == np.float32(1.0)
    assert np.array_equal(outs["L0.b"], np.array([[63.5, -32.0, 63.75, 31.5]], np.float32))


def test_chain_steps_give_run_outputs():
    """The streaming chain (accumulators, then the epilogue) yields exactly
    what the whole-chain runner gives, op by op, with each op's input being
    the previous op's int8 output."""
    import oracle.chain as chain
    import workloads as wk
    wl = wk.workloads()["c3_seq128_s80"]
    outs, scales, ins = chain.run(wl)
    calib = dict(scales)
    n = 0
    for key, wd, x, sx, kind, so, acc, y in chain.steps(wl, calib):
        xr, sxr = ins[key]
        assert np.array_equal(x, xr) and sx == sxr
        assert np.array_equal(acc, oracle.acc(xr, wd["w"]))
        assert np.array_equal(y, outs[key])
        n += 1
    assert n == len(wk.op_list(wl)) == 24
