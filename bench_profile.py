"""Turn rocprofv3 output of ``bench.py`` runs into the short summaries kept
under ``profiles/``.

    # kernel durations (rocprofv3 --kernel-trace --stats --output-format csv)
    python bench_profile.py stats --dir <rocprof dir> --bench-log <bench stdout> \
        --cmd "<the rocprofv3 command>" --out profiles/<kernel>_<workload>_kernel_trace.md

    # per-launch averages of any counters (SQ waits, issue mix) from --pmc passes
    python bench_profile.py counters --dir <dir> --log <stdout> --cmd "..." [--dir ... --log ... --cmd ...] \
        --out profiles/<kernel>_<workload>_sq_counters.md

    # HBM bytes per launch from two counter runs of bench.py --copy-calib
    python bench_profile.py traffic --fetch <dir> --fetch-log <stdout> --write <dir> --write-log <stdout> \
        --cmd-fetch "..." --cmd-write "..." --out profiles/traffic.json --md profiles/<...>.md

Dispatches of this library's kernels are matched to the bench's names by
the bench's launch order (stated in bench.py), read together with the bench
line the profiled run printed. The counters FETCH_SIZE and WRITE_SIZE
(KiB per dispatch, L2 to memory fabric) are scaled by the bytes a plain copy
of known size moves divided by what the same counter reads for it.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import bench  # noqa: E402  (constants and the kernel source hash only)
import workloads as wk  # noqa: E402


def bench_names(workload: str):
    wl = wk.workloads()[workload]
    return ["quantize_act"] + [f"L{layer}.{op.name}" for layer, op in wk.op_list(wl)]


def _is_lib_kernel(name: str) -> bool:
    return "sparse_linear" in name or "quantize_" in name


def _rows(d: str, suffix: str):
    files = sorted(glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True))
    if not files:
        raise SystemExit(f"no *{suffix} under {d}")
    out = []
    for fn in files:
        with open(fn, newline="") as f:
            out.extend(csv.DictReader(f))
    return out


def _dispatch_key(r):
    return int(r.get("Dispatch_Id") or r.get("Correlation_Id"))


def _bench_line(path):
    line = None
    with open(path) as f:
        for ln in f:
            if ln.startswith("{") and '"metric"' in ln:
                line = json.loads(ln)
    if line is None:
        raise SystemExit(f"no bench JSON line in {path}")
    return line


def _map_by_order(dispatches, names, bl):
    """dispatches: [(id, kernel_name, value)] of this library's kernels, bl:
    the bench line of the run -> ({name: [values in timed steps]},
    {name: [values in the per-kernel leg]}, {name: kernel symbol}).

    Bench launch order: one step per buffer set, W warm-up steps, K timed
    steps (each step: the n_k kernels in order), K warm steps, K in-step
    steps, then, per kernel in step order, LEG_REPLAYS replays of a graph of
    KERNEL_REPS launches."""
    dispatches = sorted(dispatches)
    n_k = len(names)
    sets, warm, steps = bl["config"]["buffer_sets"], bl["warmup"], bl["steps"]
    reps = bl["config"]["kernel_reps"] * bl["config"].get("leg_replays", 1)
    n_step = (sets + warm + 3 * steps) * n_k
    if len(dispatches) != n_step + reps * n_k:
        raise SystemExit(f"{len(dispatches)} library dispatches, expected {n_step + reps * n_k}")
    timed, leg, kname = defaultdict(list), defaultdict(list), {}
    for i, (_, name, val) in enumerate(dispatches):
        if i < n_step:
            j = i % n_k
            if sets + warm <= i // n_k < sets + warm + steps:
                timed[names[j]].append(val)
        else:
            j = (i - n_step) // reps
            leg[names[j]].append(val)
        if (j == 0) != ("quantize" in name):
            raise SystemExit(f"dispatch {i} ({name}) does not fit the launch order {names}")
        kname.setdefault(names[j], name)
    return timed, leg, kname


def cmd_stats(a):
    names = bench_names(a.workload)
    trace = _rows(a.dir, "kernel_trace.csv")
    disp = [(_dispatch_key(r), r["Kernel_Name"], (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
            for r in trace if _is_lib_kernel(r["Kernel_Name"])]
    bench_line = _bench_line(a.bench_log)
    timed, leg, kname = _map_by_order(disp, names, bench_line)
    stats = _rows(a.dir, "kernel_stats.csv")
    lines = [f"# rocprofv3 kernel trace: {a.title}", "", "Command (from the repository root):", "", "```",
             a.cmd, "```", "",
             "Per-op launch duration from the kernel trace (dispatches matched to ops by the bench's launch "
             "order) in the timed steps and in the per-kernel leg, next to the bench's own figures of the same "
             "run (in-step: the timed step's time shared out over its kernels by their legs; leg: "
             "graph-replayed launches, timed with HIP events), and the roofline fraction each gives. The "
             "profiler's per-dispatch overhead lengthens the profiled run's step, so the bench line of an "
             "unprofiled run is the one to compare fractions with:", "",
             "| op | kernel | launches (steps) | avg us (trace, steps) | avg us (bench, in-step) | trace/bench "
             "| launches (leg) | avg us (trace, leg) | avg us (bench, leg) | trace/bench | frac (trace, steps) "
             "| frac (bench, in-step) |",
             "|---|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for n in names:
        v, u = timed.get(n, []), leg.get(n, [])
        avg = sum(v) / len(v) if v else float("nan")
        avg_leg = sum(u) / len(u) if u else float("nan")
        k = bench_line["kernels"][n]
        ev, evl = k["us_instep"], k["us_leg"]
        frac_t = k["algorithmic_bytes"] / (avg * 1e-6) / 1e9 / bench.HBM_PEAK_GBS
        lines.append(f"| {n} | `{kname.get(n, '?')[:90]}` | {len(v)} | {avg:.2f} | {ev} | {avg / ev:.3f} | "
                     f"{len(u)} | {avg_leg:.2f} | {evl} | {avg_leg / evl:.3f} | {frac_t:.4f} | {k['frac_instep']} |")
    if a.ref_bench_log:
        ref = _bench_line(a.ref_bench_log)
        rk = ref["kernels"] if ref["config"]["workload"].startswith(a.workload + ":") else \
            (ref.get("workloads") or {}).get(a.workload, {}).get("kernels")
        if rk:
            lines += ["", f"Against an unprofiled run of `{a.ref_cmd}` (same kernel source; its in-step "
                          "figures, the ones the bench line reports):", "",
                      "| op | avg us (trace, steps) | us (unprofiled bench, in-step) | frac (trace) "
                      "| frac (unprofiled bench) | ratio |", "|---|---:|---:|---:|---:|---:|"]
            for n in names:
                v = timed.get(n, [])
                avg = sum(v) / len(v) if v else float("nan")
                k = bench_line["kernels"][n]
                frac_t = k["algorithmic_bytes"] / (avg * 1e-6) / 1e9 / bench.HBM_PEAK_GBS
                fb = rk[n]["frac_instep"]
                lines.append(f"| {n} | {avg:.2f} | {rk[n]['us_instep']} | {frac_t:.4f} | {fb} | {fb / frac_t:.3f} |")
    lines += ["", "rocprofv3 --stats summary (all kernels of the run, top 12 by total time):", "",
              "| kernel | calls | total ns | avg ns | min ns | max ns | % |", "|---|---:|---:|---:|---:|---:|---:|"]
    stats.sort(key=lambda r: -float(r.get("TotalDurationNs", 0)))
    for r in stats[:12]:
        lines.append(f"| `{r['Name'][:90]}` | {r['Calls']} | {r['TotalDurationNs']} | {float(r['AverageNs']):.0f} | "
                     f"{r['MinNs']} | {r['MaxNs']} | {float(r['Percentage']):.2f} |")
    lines += ["", "Bench line of the profiled run:", "", "```", json.dumps(bench_line), "```"]
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter(d, counter):
    rows = _rows(d, "counter_collection.csv")
    vals = defaultdict(float)
    kn = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        k = _dispatch_key(r)
        vals[k] += float(r["Counter_Value"])
        kn[k] = r["Kernel_Name"]
    return vals, kn


def cmd_traffic(a):
    names = bench_names(a.workload)
    res = {}
    for counter, d, log in (("FETCH_SIZE", a.fetch, a.fetch_log), ("WRITE_SIZE", a.write, a.write_log)):
        bl = _bench_line(log)
        vals, kn = _counter(d, counter)
        copies = [vals[k] for k in sorted(vals) if "bitwise_not" in kn[k]][-bench.COPY_CALIB_LAUNCHES:]
        if len(copies) != bench.COPY_CALIB_LAUNCHES:
            raise SystemExit(f"{counter}: expected {bench.COPY_CALIB_LAUNCHES} copy launches in {d}")
        copy_kib = sum(copies) / len(copies)
        scale = bench.COPY_CALIB_BYTES / (copy_kib * 1024.0)
        disp = [(k, kn[k], vals[k]) for k in vals if _is_lib_kernel(kn[k])]
        timed, _, kname = _map_by_order(disp, names, bl)
        res[counter] = {"copy_kib": copy_kib, "scale": scale, "per": timed, "kname": kname}
    kernels = {}
    for n in names:
        f = res["FETCH_SIZE"]["per"][n]
        w = res["WRITE_SIZE"]["per"][n]
        fb = sum(f) / len(f) * 1024.0 * res["FETCH_SIZE"]["scale"]
        wb = sum(w) / len(w) * 1024.0 * res["WRITE_SIZE"]["scale"]
        kernels[n] = {"kernel": res["FETCH_SIZE"]["kname"][n], "launches": len(f),
                      "fetch_bytes": round(fb), "write_bytes": round(wb), "hbm_bytes_per_launch": round(fb + wb)}
    out = {"kernel_source_sha256_16": bench.kernel_source_hash(), "workload": a.workload,
           "copy_calib": {"bytes_each_way": bench.COPY_CALIB_BYTES,
                          "fetch_size_kib": res["FETCH_SIZE"]["copy_kib"], "fetch_scale": res["FETCH_SIZE"]["scale"],
                          "write_size_kib": res["WRITE_SIZE"]["copy_kib"], "write_scale": res["WRITE_SIZE"]["scale"]},
           "command_fetch": a.cmd_fetch, "command_write": a.cmd_write, "kernels": kernels}
    with open(a.out, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    if a.md:
        lines = [f"# HBM traffic per launch: {a.title}", "", "Counter runs (from the repository root):", "", "```",
                 a.cmd_fetch, a.cmd_write, "```", "",
                 f"Scale: a plain copy of {bench.COPY_CALIB_BYTES} bytes reads FETCH_SIZE = "
                 f"{res['FETCH_SIZE']['copy_kib']:.0f} KiB (factor {res['FETCH_SIZE']['scale']:.4f}) and WRITE_SIZE = "
                 f"{res['WRITE_SIZE']['copy_kib']:.0f} KiB (factor {res['WRITE_SIZE']['scale']:.4f}).", "",
                 "| op | launches | fetch MB | write MB | total MB per launch |", "|---|---:|---:|---:|---:|"]
        for n, k in kernels.items():
            lines.append(f"| {n} | {k['launches']} | {k['fetch_bytes'] / 1e6:.3f} | {k['write_bytes'] / 1e6:.3f} | "
                         f"{k['hbm_bytes_per_launch'] / 1e6:.3f} |")
        lines += ["", f"Kernel source sha256[:16] = {out['kernel_source_sha256_16']}"]
        with open(a.md, "w") as f:
            f.write("\n".join(lines) + "\n")
        print("\n".join(lines))


def cmd_counters(a):
    """Average of each counter per launch of each op over the timed steps,
    from one or more --pmc runs of bench.py (each pass its own directory and
    stdout), with the wave-time shares of the SQ wait and issue counters."""
    names = bench_names(a.workload)
    avg = defaultdict(dict)
    for d, log in zip(a.dir, a.log):
        bl = _bench_line(log)
        counters = sorted({r["Counter_Name"] for r in _rows(d, "counter_collection.csv")})
        for c in counters:
            vals, kn = _counter(d, c)
            disp = [(k, kn[k], vals[k]) for k in vals if _is_lib_kernel(kn[k])]
            timed, _, _ = _map_by_order(disp, names, bl)
            for n in names:
                v = timed.get(n, [])
                if v:
                    avg[n][c] = sum(v) / len(v)
    lines = [f"# rocprofv3 counters: {a.title}", "", "Counter runs (from the repository root):", "", "```", *a.cmd,
             "```", "", "Average per launch over the timed steps (SQ wave counters count units of 4 cycles, summed "
             "over waves; SQ_VALU_MFMA_BUSY_CYCLES counts SIMD cycles):", ""]
    counters = sorted({c for n in names for c in avg[n]})
    lines += ["| counter | " + " | ".join(names) + " |", "|---|" + "---:|" * len(names)]
    for c in counters:
        lines.append(f"| {c} | " + " | ".join(f"{avg[n].get(c, float('nan')):.0f}" for n in names) + " |")
    shares = [k for k in ("SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_VALU",
                          "SQ_ACTIVE_INST_SCA", "SQ_ACTIVE_INST_LDS", "SQ_ACTIVE_INST_VMEM")]
    lines += ["", "Share of SQ_WAVE_CYCLES:", "", "| counter | " + " | ".join(names) + " |",
              "|---|" + "---:|" * len(names)]
    for c in shares:
        row = []
        for n in names:
            wc = avg[n].get("SQ_WAVE_CYCLES")
            row.append(f"{100.0 * avg[n][c] / wc:.1f} %" if wc and c in avg[n] else "-")
        lines.append(f"| {c} | " + " | ".join(row) + " |")
    lines += ["", f"Kernel source sha256[:16] = {bench.kernel_source_hash()}"]
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    p = argparse.ArgumentParser()
    sub = p.add_subparsers(dest="what", required=True)
    s = sub.add_parser("stats")
    s.add_argument("--dir", required=True)
    s.add_argument("--bench-log", required=True)
    s.add_argument("--cmd", required=True)
    s.add_argument("--out", required=True)
    s.add_argument("--title", default="")
    s.add_argument("--workload", default="c1")
    s.add_argument("--ref-bench-log", help="stdout of an unprofiled bench.py run to compare fractions with")
    s.add_argument("--ref-cmd", default="python bench.py")
    c = sub.add_parser("counters")
    c.add_argument("--dir", action="append", required=True, help="rocprof directory of one --pmc pass (repeat)")
    c.add_argument("--log", action="append", required=True, help="stdout of that pass (holds the bench line)")
    c.add_argument("--cmd", action="append", required=True, help="the rocprofv3 command of that pass")
    c.add_argument("--out", required=True)
    c.add_argument("--title", default="")
    c.add_argument("--workload", default="c1")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--fetch-log", required=True, help="stdout of the FETCH_SIZE run (holds the bench line)")
    t.add_argument("--write-log", required=True)
    t.add_argument("--cmd-fetch", required=True)
    t.add_argument("--cmd-write", required=True)
    t.add_argument("--out", required=True)
    t.add_argument("--md")
    t.add_argument("--title", default="")
    t.add_argument("--workload", default="c1")
    a = p.parse_args()
    {"stats": cmd_stats, "traffic": cmd_traffic, "counters": cmd_counters}[a.what](a)


if __name__ == "__main__":
    main()
