"""Host logic of the benchmark and of the profile summariser, on the CPU:
the one-GPU contract, the per-kernel table's arithmetic, the roofline bound
choice, and the mapping of profiler dispatches to ops by launch order (which
must follow the bench's sequence of passes)."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import bench_profile  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"]


def test_bound_follows_the_published_peaks():
    # c1 FFN1: 16.11 MB and 1.933 GOP -> HBM (2.01 us against 0.39 us)
    assert bench._bound(16.11e6, 1.933e9) == "hbm"
    # an op-heavy launch with few bytes is matrix-bound
    assert bench._bound(1e6, 1e12) == "mfma"
    # the balance point: bytes / 8 TB/s == ops / 5 POP/s
    assert bench._bound(8e6, 5e9) == "hbm"


class _FakeRunner:
    names = ["quantize_act", "L0.ffn1", "L0.ffn2"]
    kbytes = [15.73e6, 16.11e6, 25.53e6]
    kops = [0.0, 1.933e9, 1.933e9]


def test_kernel_table_shares_the_step_by_the_legs():
    legs = np.array([4.0, 15.0, 15.0])
    ms_step = 0.0375  # 37.5 us: legs sum to 34 us, so each gets 37.5/34 of its leg
    t = bench.kernel_table(_FakeRunner(), legs, ms_step, None, 5000.0)
    share = 37.5 / 34.0
    assert sum(t[n]["us_instep"] for n in _FakeRunner.names) == pytest.approx(37.5, abs=2e-3)
    for j, n in enumerate(_FakeRunner.names):
        e = t[n]
        assert e["bound"] == "hbm"
        assert e["us_leg"] == pytest.approx(legs[j])
        assert e["us_instep"] == pytest.approx(legs[j] * share, abs=1e-3)
        gbs = _FakeRunner.kbytes[j] / (e["us_instep"] * 1e-6) / 1e9
        assert e["hbm_GBs_instep"] == pytest.approx(gbs, rel=1e-3)
        assert e["frac_instep"] == pytest.approx(gbs / bench.HBM_PEAK_GBS, abs=1e-4)
        assert e["frac_vs_copy"] == pytest.approx(gbs / 5000.0, abs=1e-4)
        assert e["tops_leg"] == pytest.approx(_FakeRunner.kops[j] / (legs[j] * 1e-6) / 1e12, rel=1e-3)


def test_kernel_source_hash_is_16_hex_digits_and_stable():
    h = bench.kernel_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0
    assert bench.kernel_source_hash() == h


def _bench_line(sets, warm, steps, reps, replays):
    return {"warmup": warm, "steps": steps,
            "config": {"buffer_sets": sets, "kernel_reps": reps, "leg_replays": replays}}


def test_dispatches_map_to_ops_by_the_bench_launch_order():
    names = ["quantize_act", "L0.ffn1", "L0.ffn2"]
    kern = ["quantize_t16x32_kernel", "sparse_linear_panel_gelu_kernel", "sparse_linear_direct_kernel"]
    sets, warm, steps, reps, replays = 3, 2, 4, 5, 2
    disp, i = [], 0
    # one step per buffer set, warm-up, timed, warm, in-step: (sets + warm + 3 steps) steps of all ops
    for s in range(sets + warm + 3 * steps):
        for j in range(3):
            timed = sets + warm <= s < sets + warm + steps
            disp.append((i, kern[j], 100.0 + j if timed else 1.0))
            i += 1
    # then each op's leg: replays x reps launches
    for j in range(3):
        for _ in range(reps * replays):
            disp.append((i, kern[j], 10.0 + j))
            i += 1
    timed, leg, kname = bench_profile._map_by_order(disp, names, _bench_line(sets, warm, steps, reps, replays))
    for j, n in enumerate(names):
        assert timed[n] == [100.0 + j] * steps
        assert leg[n] == [10.0 + j] * (reps * replays)
        assert kname[n] == kern[j]


def test_dispatch_count_mismatch_is_refused():
    names = ["quantize_act", "L0.ffn1"]
    disp = [(i, "quantize_t16x32_kernel" if i % 2 == 0 else "sparse_linear_kernel", 1.0) for i in range(10)]
    with pytest.raises(SystemExit):
        bench_profile._map_by_order(disp, names, _bench_line(1, 1, 1, 1, 1))
