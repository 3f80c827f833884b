"""Oracle-side runner for chains of sparse linears -- TEST INFRASTRUCTURE ONLY.

Runs a workload's ops in order with the CPU oracle: an op's input is either
its seeded int8 activations or the int8 output of an earlier op (whose
calibrated output scale becomes this op's activation scale). Output scales of
int8 ops are calibrated as so = max|g| / 127 over the op's fp32 pre-requant
output g on the full seed-0 batch.

Because token rows never mix inside a linear, the chain can also be run on any
subset of rows (``rows=``) with scales taken from a stored calibration, which
gives exact oracle values for sampled outputs of very large batches.
"""
from __future__ import annotations

from typing import Dict, Iterator, Optional, Sequence

import numpy as np

import oracle
import workloads as wk

_F32_OF = {"i8": oracle.KIND_F32, "i8_gelu": oracle.KIND_F32_GELU,
           "f32": oracle.KIND_F32, "f32_gelu": oracle.KIND_F32_GELU}
_KIND = {"f32": oracle.KIND_F32, "f32_gelu": oracle.KIND_F32_GELU,
         "i8": oracle.KIND_I8, "i8_gelu": oracle.KIND_I8_GELU}


def op_key(layer: int, name: str) -> str:
    return f"L{layer}.{name}"


def steps(wl: wk.Workload, calib: Dict[str, float], seed: int = 0) -> Iterator[tuple]:
    """The chain one op at a time with stored output scales, holding only the
    outputs a later op still reads (for very large batches). Yields
    (key, x, sx, kind, so, acc, y): the op's int8 input and its scale, the
    oracle kind, the output scale (1.0 for fp32 kinds), the int32
    accumulators and the final output. The layer is the contraction followed
    by the epilogue (Section "Sparse GEMM operators"), so y is computed from
    acc by the oracle's epilogue: the same values oracle.linear gives."""
    later = {wl.op_src(l2, o2) for l2, o2 in wk.op_list(wl)} - {"seeded"}
    outs: Dict[str, np.ndarray] = {}
    for layer, op in wk.op_list(wl):
        key = op_key(layer, op.name)
        src = wl.op_src(layer, op)
        if src == "seeded":
            x, sx = wk.op_seeded_x(wl, layer, op, seed=seed), float(wk.SX)
        else:
            x, sx = outs[src], float(calib[src])
        wd = wk.op_weight(wl, layer, op, seed=seed)
        kname = wl.op_kind(layer, op)
        so = float(calib[key]) if kname in ("i8", "i8_gelu") else 1.0
        acc = oracle.acc(x, wd["w"])
        y = oracle.epilogue(acc, sx, wd["sw"], wd["b"], _KIND[kname], so=so)
        if key in later:
            outs[key] = y
        yield key, wd, x, sx, _KIND[kname], so, acc, y
        del acc


def run(wl: wk.Workload, calib: Optional[Dict[str, float]] = None, rows: Optional[Sequence[int]] = None,
        seed: int = 0, keep_outputs: bool = True, weights: Optional[Dict[str, dict]] = None):
    """Run the chain. Returns (outputs, scales, inputs).

    calib None: calibrate every int8 op's scale on the (full) batch.
    calib given: use the stored scales (required when rows is a subset).
    outputs[key] is the op's final output (int8 or fp32); inputs[key] = (x, sx).
    """
    if calib is None and rows is not None:
        raise ValueError("calibration needs the full batch")
    scales: Dict[str, float] = {}
    outs: Dict[str, np.ndarray] = {}
    ins: Dict[str, tuple] = {}
    for layer, op in wk.op_list(wl):
        key = op_key(layer, op.name)
        src = wl.op_src(layer, op)
        if src == "seeded":
            x = wk.op_seeded_x(wl, layer, op, seed=seed)
            if rows is not None:
                x = x[np.asarray(rows)]
            sx = float(wk.SX)
        else:
            x = outs[src]
            sx = scales[src]
        wd = weights[key] if weights is not None else wk.op_weight(wl, layer, op, seed=seed)
        kind = wl.op_kind(layer, op)
        if kind in ("i8", "i8_gelu"):
            if calib is None:
                g = oracle.linear(x, wd["w"], sx, wd["sw"], wd["b"], _F32_OF[kind])
                so = float(oracle.calibrate_out_scale(g))
                y = oracle.quantize(g, so)
                del g
            else:
                so = float(calib[key])
                y = oracle.linear(x, wd["w"], sx, wd["sw"], wd["b"], _KIND[kind], so=so)
            scales[key] = so
        else:
            y = oracle.linear(x, wd["w"], sx, wd["sw"], wd["b"], _KIND[kind])
        ins[key] = (x, sx)
        outs[key] = y
        if not keep_outputs:
            # keep only what a later op still reads
            needed = set()
            for l2, o2 in wk.op_list(wl):
                s2 = wl.op_src(l2, o2)
                if s2 != "seeded":
                    needed.add(s2)
            for k in list(outs):
                if k not in needed and k != key:
                    del outs[k]
            for k in list(ins):
                if k != key:
                    del ins[k]
    return outs, scales, ins
