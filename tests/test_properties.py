"""Property tests on the CPU (hypothesis, derandomised): the packer's canonical
form and GPU tile image against the dense weight, and the oracle against
pure-Python brute force, over generated shapes, masks and values.

* packing: unpack(pack(W)) == W; the exported BSR lists exactly the 4x1
  blocks with a non-zero value, columns ascending, values in place; the tile
  statistics agree with the shape;
* oracle: int32 accumulators equal the integer sum written out; the fp32
  epilogue equals the three separately rounded fp32 operations of its
  definition.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import paper_2211_07715_amd as sl

SETTINGS = settings(max_examples=60, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow])


@st.composite
def block_sparse_weight(draw):
    n = 4 * draw(st.integers(1, 24))
    k = draw(st.integers(1, 300))
    density = draw(st.sampled_from([0.0, 0.02, 0.1, 0.3, 0.7, 1.0]))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    rng = np.random.default_rng(seed)
    keep = rng.random((n // 4, k)) < density
    # some block-rows get a run of consecutive blocks, so that aligned groups
    # of 4 columns with 3 or 4 blocks (the overflow operands) appear
    if draw(st.booleans()) and k >= 4:
        g = rng.integers(0, n // 4)
        c0 = 4 * rng.integers(0, k // 4)
        keep[g, c0:c0 + 4] = True
    w = rng.integers(-127, 128, size=(n, k), dtype=np.int8)
    if draw(st.booleans()):
        w[rng.random((n, k)) < 0.2] = 0  # zero values inside stored blocks
    return (w * np.repeat(keep, 4, axis=0).astype(np.int8)).astype(np.int8)


@SETTINGS
@given(block_sparse_weight())
def test_pack_round_trips(w):
    n, k = w.shape
    sw = np.full(n, 0.005, np.float32)
    pw = sl.PackedWeight.pack(w, sw, None, host_only=True)
    try:
        assert np.array_equal(pw.unpack(), w)
        row_ptr, col, vals = pw.export_bsr()
        blocks = w.reshape(n // 4, 4, k)
        stored = np.any(blocks != 0, axis=1)  # [n/4, k]
        assert row_ptr[0] == 0 and np.all(np.diff(row_ptr.astype(np.int64)) >= 0)
        assert int(row_ptr[-1]) == int(stored.sum()) == pw.nnz_blocks()
        for g in range(n // 4):
            cols = col[row_ptr[g]:row_ptr[g + 1]].astype(np.int64)
            assert np.array_equal(cols, np.nonzero(stored[g])[0])
            assert np.array_equal(vals[row_ptr[g]:row_ptr[g + 1]], blocks[g][:, cols].T)
        stats = pw.tile_stats()
        assert stats["n_tiles"] == (n + 15) // 16
        assert 0 <= stats["n_overflow"] <= stats["n_entries"]
        if stored.sum() == 0:
            assert stats["n_entries"] == 0
    finally:
        pw.free()


@SETTINGS
@given(st.integers(1, 4), st.integers(1, 3), st.integers(1, 9), st.integers(0, 2 ** 31 - 1),
       st.booleans())
def test_oracle_matches_brute_force(m, n4, k, seed, extremes):
    rng = np.random.default_rng(seed)
    n = 4 * n4
    if extremes:
        x = rng.choice(np.array([-127, -1, 0, 1, 127], np.int8), size=(m, k))
        w = rng.choice(np.array([-127, -1, 0, 1, 127], np.int8), size=(n, k))
    else:
        x = rng.integers(-127, 128, (m, k), dtype=np.int8)
        w = rng.integers(-127, 128, (n, k), dtype=np.int8)
    sw = rng.uniform(0.001, 0.01, n).astype(np.float32)
    b = rng.normal(0, 0.02, n).astype(np.float32)
    sx = np.float32(0.02)
    got = oracle.acc(x, w)
    ref = [[sum(int(x[i, kk]) * int(w[j, kk]) for kk in range(k)) for j in range(n)] for i in range(m)]
    assert np.array_equal(got, np.array(ref, dtype=np.int64))
    y = oracle.linear(x, w, float(sx), sw, b, oracle.KIND_F32)
    for i in range(m):
        for j in range(n):
            s = np.float32(sx * sw[j])
            want = np.float32(np.float32(np.float32(ref[i][j]) * s) + b[j])
            assert y[i, j] == want, (i, j, y[i, j], want)
