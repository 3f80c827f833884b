"""Benchmark of the sparse INT8 linear path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c1]

Workload (default): the DistilBERT FFN pair at batch 32 x seq 128 (M = 4096
tokens), 4x1 block sparsity 90 %: W1 3072x768 (dequant + bias + GELU(erf) +
requant to int8), W2 768x3072 (dequant + bias to fp32).

One step is one pass of the whole hot path over one batch: quantize_act of the
fp32 input -> linear 1 (int8 out) -> linear 2 (fp32 out), all on one stream.
The int8 activations between them stay in the library's 16-token x
32-feature block layout (--layout t16x32, the default: the order the matrix
cores read; the quantisation writes it and linear 1 writes its int8 output in
it), or are row-major throughout (--layout rows).
Inputs are resident in HBM when timing starts; the step rotates over enough
input/output buffer sets (> 2x the 256 MB last-level cache) that every step
reads its activations from HBM, not from a cache warmed by the previous step.

Prints ONE JSON line. ``value`` is effective int8 TOPS over non-zero MACs
(2 * M * 4 * stored_blocks per linear, summed) per step time; the K timed
steps are bracketed by two HIP events on the launch stream. Afterwards each
kernel of the step is launched KERNEL_REPS times back to back (same rotating
buffers) from a captured HIP graph, between two events, which gives its
average launch duration free of host launch cost.
``roofline`` describes the slowest kernel against the HBM bound: its
algorithmic bytes (X + Y + canonical packed W + scales) per launch divided by
that duration; ``traffic`` is the counter-measured bytes per launch from
profiles/traffic.json when that file was taken on the current kernel source.
``cpu_baseline`` times the CPU oracle on the same step. ``layer_latency``
gives the DistilBERT-layer latency: one layer's four linears at batch 32 x
seq 128 and the 6-layer stack at batch 1 x seq 128 (80 % sparsity, warm,
host-launched and replayed from a HIP graph).

Launch order (used to match profiler dispatches to ops): one step per buffer
set (set-up), W warm-up steps, K timed steps, then, per kernel in step order,
LEG_REPLAYS replays of a graph of KERNEL_REPS launches; with --copy-calib,
three elementwise copies last.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, published
MFMA_I8_PEAK_TOPS = 5000.0   # MI355X dense int8 matrix peak, published
MALL_BYTES = 256 << 20
COPY_CALIB_BYTES = 256 << 20  # one read and one write of this many bytes per copy launch
COPY_CALIB_LAUNCHES = 3
KERNEL_REPS = 50  # launches per kernel in the per-kernel timing leg (one graph)
LEG_REPLAYS = 2   # replays of each kernel's graph; the last one is timed
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2211_07715_amd", "csrc", f)
                  for f in ("kernels.hip", "kernels_direct.hip", "kernels_panel.hip", "sl_device.h", "gelu_table.cpp")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for fn in KERNEL_SOURCES:
        with open(fn, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def act_shape(sl, layout, rows, cols):
    """Device shape of an int8 activation in the chosen layout."""
    return sl.t16x32_shape(rows, cols) if layout == sl.LAYOUT_T16X32 else (rows, cols)


def algorithmic_bytes(m, n, k, nnzb, out_bytes):
    """X + Y + canonical packed W (4 B values + 2 B column per block, row
    pointers) + per-channel scale and bias."""
    return m * k + m * n * out_bytes + nnzb * 6 + (n // 4 + 1) * 4 + 8 * n


def chain_latency(torch, sl, wk, name, calib, stream, dev, layout, reps=200, warmup=20):
    """Latency of a workload's chain of linears (inputs resident, buffers
    reused: a warm, latency-oriented figure). Returns host-launched time per
    chain and per layer, and the same chain replayed from a HIP graph (after
    checking that a replay reproduces the eagerly computed outputs)."""
    wl = wk.workloads()[name]
    ops = wk.op_list(wl)
    packed, bufs, seeded, kinds = {}, {}, {}, {}
    for layer, op in ops:
        key = f"L{layer}.{op.name}"
        wd = wk.op_weight(wl, layer, op)
        packed[key] = sl.PackedWeight.pack(wd["w"], wd["sw"], wd["b"])
        kinds[key] = sl.EPI_BY_NAME[wl.op_kind(layer, op)]
        dt = torch.int8 if kinds[key] in (3, 4) else (torch.int32 if kinds[key] == 0 else torch.float32)
        shape = act_shape(sl, layout, wl.m, op.n_out) if kinds[key] in (3, 4) else (wl.m, op.n_out)
        bufs[key] = torch.empty(shape, dtype=dt, device=dev)
        if wl.op_src(layer, op) == "seeded":
            xs8 = wk.op_seeded_x(wl, layer, op)
            if layout == sl.LAYOUT_T16X32:
                xs8 = sl.to_t16x32(xs8)
            seeded[key] = torch.from_numpy(xs8).to(dev)

    def chain():
        st = torch.cuda.current_stream()  # the capture stream while a graph is recorded
        for layer, op in ops:
            key = f"L{layer}.{op.name}"
            src = wl.op_src(layer, op)
            if src == "seeded":
                xin, xs = seeded[key], float(wk.SX)
            else:
                xin, xs = bufs[src], float(calib[src])
            yl = layout if kinds[key] in (3, 4) else sl.LAYOUT_ROWS
            packed[key].run(xin, xs, kinds[key], out_scale=float(calib.get(key, 1.0)), out=bufs[key], stream=st,
                            x_layout=layout, y_layout=yl, m_tokens=wl.m)

    for _ in range(warmup):
        chain()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        chain()
    e1.record(stream)
    torch.cuda.synchronize()
    eager_us = e0.elapsed_time(e1) / reps * 1e3
    out = {"workload": f"{wl.name}: {wl.notes}", "m_tokens": wl.m, "layers": wl.layers, "linears": len(ops),
           "activation_layout": "t16x32" if layout == sl.LAYOUT_T16X32 else "rows",
           "chain_us": round(eager_us, 2), "per_layer_us": round(eager_us / wl.layers, 2)}
    ref = {k: v.clone() for k, v in bufs.items()}
    try:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            chain()
        ok = True
        for _ in range(3):
            for v in bufs.values():
                v.zero_()
            g.replay()
            torch.cuda.synchronize()
            ok = ok and all(torch.equal(bufs[k], ref[k]) for k in bufs)
            chain()  # eager work between replays
            torch.cuda.synchronize()
        if ok:
            for _ in range(warmup):
                g.replay()
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(reps):
                g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            gus = e0.elapsed_time(e1) / reps * 1e3
            out["graph_chain_us"] = round(gus, 2)
            out["graph_per_layer_us"] = round(gus / wl.layers, 2)
        else:
            out["graph_chain_us"] = None
            out["graph_note"] = "graph replay did not reproduce the eager outputs"
    except Exception as e:  # graph capture unavailable: report the eager figure only
        out["graph_chain_us"] = None
        out["graph_note"] = f"graph capture failed: {type(e).__name__}"
    for w in packed.values():
        w.free()
    return out


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default="c1")
    p.add_argument("--layout", choices=("t16x32", "rows"), default="t16x32",
                   help="layout of the int8 activations between the kernels")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    p.add_argument("--cpu-seconds", type=float, default=10.0)
    p.add_argument("--no-latency", action="store_true", help="skip the DistilBERT-layer latency legs")
    p.add_argument("--copy-calib", action="store_true",
                   help="after the timed steps, run a plain elementwise copy of COPY_CALIB_BYTES three times "
                        "(the reference kernel that scales the HBM byte counters)")
    return p.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}), flush=True)
        sys.exit(2)

    import torch
    import paper_2211_07715_amd as sl
    import workloads as wk

    sl.load()  # fails loudly without the HIP library
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}), flush=True)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layout = sl.LAYOUT_T16X32 if args.layout == "t16x32" else sl.LAYOUT_ROWS

    wl = wk.workloads()[args.workload]
    with open(os.path.join(ROOT, "tests", "golden", "calibration.json")) as f:
        calib = json.load(f)[wl.name]
    ops = wk.op_list(wl)
    if wl.layers != 1:
        raise SystemExit("bench workloads are single-layer op chains")

    # ---- weights (packed once, offline)
    packed, meta = [], []
    for layer, op in ops:
        key = f"L{layer}.{op.name}"
        wd = wk.op_weight(wl, layer, op)
        pw = sl.PackedWeight.pack(wd["w"], wd["sw"], wd["b"])
        kind = sl.EPI_BY_NAME[wl.op_kind(layer, op)]
        src = wl.op_src(layer, op)
        meta.append(dict(key=key, n=op.n_out, k=op.k_in, kind=kind, src=src,
                         so=float(calib.get(key, 1.0)), nnzb=pw.nnz_blocks(), stats=pw.tile_stats()))
        packed.append(pw)
    first = ops[0][1]
    m = wl.m

    # ---- activations: fp32 input whose quantisation is the seeded int8 X
    sx = np.float32(wk.SX)
    x_i8 = wk.op_seeded_x(wl, ops[0][0], first)
    x_f32 = (x_i8.astype(np.float32) * sx).astype(np.float32)
    out_bytes = {0: 4, 1: 4, 2: 4, 3: 1, 4: 1}
    set_bytes = x_f32.nbytes + x_i8.nbytes + sum(m * md["n"] * out_bytes[md["kind"]] for md in meta)
    n_sets = max(2, int(np.ceil(2.2 * MALL_BYTES / set_bytes)))
    sets = []
    xf_dev = torch.from_numpy(x_f32).to(dev)
    for _ in range(n_sets):
        s = {"xf": xf_dev.clone(), "q": torch.empty(act_shape(sl, layout, m, first.k_in), dtype=torch.int8, device=dev)}
        for md in meta:
            dt = {0: torch.int32, 1: torch.float32, 2: torch.float32, 3: torch.int8, 4: torch.int8}[md["kind"]]
            shape = act_shape(sl, layout, m, md["n"]) if md["kind"] in (3, 4) else (m, md["n"])
            s[md["key"]] = torch.empty(shape, dtype=dt, device=dev)
        sets.append(s)
    del xf_dev
    stream = torch.cuda.current_stream()

    def step(s, only=None, stream=stream):
        # only=j launches just kernel j of the step (0: quantize_act, 1..: the linears)
        if only is None or only == 0:
            sl.quantize_act(s["xf"], float(sx), out=s["q"], stream=stream, layout=layout)
        for i, (pw, md) in enumerate(zip(packed, meta)):
            if only is not None and only != i + 1:
                continue
            if md["src"] == "seeded":
                xin, xs = s["q"], float(sx)
            else:
                src = md["src"]
                xin = s[src]
                xs = next(mm["so"] for mm in meta if mm["key"] == src)
            yl = layout if md["kind"] in (3, 4) else sl.LAYOUT_ROWS
            pw.run(xin, xs, md["kind"], out_scale=md["so"], out=s[md["key"]], stream=stream, x_layout=layout,
                   y_layout=yl, m_tokens=m)

    n_k = 1 + len(meta)
    # every buffer set gets valid activations once (set-up, not warm-up)
    for s in sets:
        step(s)
    for i in range(args.warmup):
        step(sets[i % n_sets])
    torch.cuda.synchronize()

    # ---- timed region: K whole steps, events only around the region
    e_start, e_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e_start.record(stream)
    for i in range(args.steps):
        step(sets[i % n_sets])
    e_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = e_start.elapsed_time(e_end) / args.steps

    # ---- per-kernel launch duration: each kernel of the step alone, KERNEL_REPS
    # launches back to back over the rotating buffer sets, captured in a HIP
    # graph (host launch cost would otherwise hide a kernel shorter than it);
    # the graph is replayed LEG_REPLAYS times and the last replay is timed
    # with HIP events on the stream it runs on
    per_kernel_us = np.zeros(n_k)
    cap = torch.cuda.Stream()
    for j in range(n_k):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            for i in range(KERNEL_REPS):
                step(sets[i % n_sets], only=j, stream=cap)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(cap):
            for r in range(LEG_REPLAYS):
                if r == LEG_REPLAYS - 1:
                    ev0.record(cap)
                g.replay()
            ev1.record(cap)
        torch.cuda.synchronize()
        per_kernel_us[j] = ev0.elapsed_time(ev1) / KERNEL_REPS * 1e3
        del g

    # ---- metric
    total_ops = sum(2 * m * 4 * md["nnzb"] for md in meta)
    tops = total_ops / (ms_per_step * 1e-3) / 1e12
    names = ["quantize_act"] + [md["key"] for md in meta]
    kbytes = [x_f32.nbytes + x_i8.nbytes] + [algorithmic_bytes(m, md["n"], md["k"], md["nnzb"], out_bytes[md["kind"]])
                                             for md in meta]
    kops = [0] + [2 * m * 4 * md["nnzb"] for md in meta]
    kernels = {}
    for j in range(n_k):
        kernels[names[j]] = {"us": round(float(per_kernel_us[j]), 3),
                             "hbm_GBs": round(kbytes[j] / (per_kernel_us[j] * 1e-6) / 1e9, 1),
                             "tops": round(kops[j] / (per_kernel_us[j] * 1e-6) / 1e12, 2)}
    dom = int(np.argmax(per_kernel_us))
    achieved = kbytes[dom] / (per_kernel_us[dom] * 1e-6) / 1e9
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if tr.get("kernel_source_sha256_16") == kernel_source_hash() and names[dom] in tr.get("kernels", {}):
            traffic = tr["kernels"][names[dom]]["hbm_bytes_per_launch"]
    roofline = {"bound": "hbm", "kernel": names[dom], "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "algorithmic_bytes": int(kbytes[dom])}

    if args.copy_calib:
        src = torch.randint(0, 256, (COPY_CALIB_BYTES,), dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(COPY_CALIB_LAUNCHES):
            torch.bitwise_not(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # ---- DistilBERT-layer latency: one layer's four linears at batch 32 x
    # seq 128, and the 6-layer stack at batch 1 x seq 128 (80 % sparsity)
    latency = None
    if not args.no_latency:
        with open(os.path.join(ROOT, "tests", "golden", "calibration.json")) as f:
            calib_all = json.load(f)
        latency = {}
        for name, label in (("c2", "bs32_seq128_80pct_layer"), ("c3_seq128_s80", "bs1_seq128_80pct_6layers")):
            latency[label] = chain_latency(torch, sl, wk, name, calib_all[name], stream, dev, layout)

    # ---- CPU oracle baseline on the same step (bounded by time)
    cpu = None
    if not args.no_cpu:
        import oracle
        ws = [wk.op_weight(wl, layer, op) for layer, op in ops]
        reps, t_cpu = 0, 0.0
        while t_cpu < args.cpu_seconds and reps < 50:
            c0 = time.perf_counter()
            q = oracle.quantize(x_f32, sx)
            outs = {}
            for (layer, op), wd, md in zip(ops, ws, meta):
                if md["src"] == "seeded":
                    xin, xs = q, float(sx)
                else:
                    xin = outs[md["src"]]
                    xs = next(mm["so"] for mm in meta if mm["key"] == md["src"])
                outs[md["key"]] = oracle.linear(xin, wd["w"], xs, wd["sw"], wd["b"], md["kind"], so=md["so"])
            t_cpu += time.perf_counter() - c0
            reps += 1
        cpu = {"value": round(total_ops * reps / t_cpu / 1e12, 5), "unit": "TOPS", "cores": oracle.threads(),
               "kind": "oracle",
               "sample": f"{reps} full step(s) of {wl.name} ({m} tokens; quantize + {len(meta)} linears, dense "
                         f"naive int32 matmul), {t_cpu:.1f} s",
               "ms_per_step": round(t_cpu / reps * 1e3, 1)}

    line = {
        "metric": "effective int8 TOPS (nonzero MACs) + % roofline; DistilBERT-layer latency @bs1/bs32",
        "value": round(tops, 3),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.notes}", "m_tokens": m,
                   "ops": [f"{md['key']} {md['n']}x{md['k']} kind={md['kind']} nnzb={md['nnzb']}" for md in meta],
                   "activation_layout": args.layout, "buffer_sets": n_sets, "kernel_reps": KERNEL_REPS, "leg_replays": LEG_REPLAYS,
                   "wall_s": round(wall, 3)},
        "kernels": kernels,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "layer_latency": latency,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
