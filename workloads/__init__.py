"""Seeded synthetic inputs for the sparse INT8 linear layer.

This module only draws random numbers and describes workload shapes. It holds
none of the layer's arithmetic (no contraction, dequantisation, GELU or
requantisation): both the CPU oracle (``oracle/``) and the HIP path are fed
from it, and neither shares anything else.

Shapes follow a DistilBERT encoder layer (hidden 768, fused QKV 2304, FFN 3072)
and a BERT-large FFN (1024 / 4096). The sparsity pattern is the paper's
block-wise structured sparsity: 1-D blocks of 4 consecutive output rows at one
input column (Appendix "Block-wise structured sparsity"; Section "Sparse GEMM
operators", constant block size 4). Which blocks survive is drawn uniformly at
random here; the paper's trained masks (average-magnitude pruning) need its
datasets and weights, which synthetic masks of the same density stand in for.

Conventions: X is ``[M x K]`` int8 (tokens x input features), W is ``[N x K]``
int8 (output x input features), Y is ``[M x N]``.

Random stream: ``numpy.random.default_rng([seed, cfg, variant, layer, op,
role])`` (PCG64) with roles 0 = block mask permutation, 1 = W values,
2 = per-channel weight scale, 3 = bias, 4 = activations.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

# per-tensor activation scale of every seeded int8 input
SX = np.float32(0.02)

ROLE_MASK, ROLE_W, ROLE_SW, ROLE_B, ROLE_X = 0, 1, 2, 3, 4

# epilogue kinds, numbered as in include/sparse_linear.h
KIND_ACC_I32, KIND_F32, KIND_F32_GELU, KIND_I8, KIND_I8_GELU = 0, 1, 2, 3, 4
KIND_NAMES = {"acc_i32": 0, "f32": 1, "f32_gelu": 2, "i8": 3, "i8_gelu": 4}


def _rng(seed: int, cfg: int, variant: int, layer: int, op: int, role: int):
    return np.random.default_rng([seed, cfg, variant, layer, op, role])


def block_keep_mask(n_out: int, k_in: int, sparsity: float, rng) -> np.ndarray:
    """Boolean ``[n_out/4, k_in]``: True where the 4x1 block survives.

    Exactly ``round(sparsity * n_blocks)`` blocks are zeroed, picked by one
    seeded permutation over all blocks of the matrix, so the number of
    surviving blocks per block-row varies.
    """
    if n_out % 4:
        raise ValueError("n_out must be a multiple of the block height 4")
    nb = (n_out // 4) * k_in
    n_zero = int(np.floor(sparsity * nb + 0.5))
    keep = np.ones(nb, dtype=bool)
    keep[rng.permutation(nb)[:n_zero]] = False
    return keep.reshape(n_out // 4, k_in)


def make_weight(n_out: int, k_in: int, sparsity: float, *, seed: int = 0, cfg: int = 0,
                variant: int = 0, layer: int = 0, op: int = 0) -> Dict[str, np.ndarray]:
    """Dense int8 W with 4x1 block sparsity, fp32 per-channel scale and bias."""
    keep = block_keep_mask(n_out, k_in, sparsity, _rng(seed, cfg, variant, layer, op, ROLE_MASK))
    w = _rng(seed, cfg, variant, layer, op, ROLE_W).integers(-127, 128, size=(n_out, k_in), dtype=np.int8)
    w *= np.repeat(keep, 4, axis=0).astype(np.int8)
    sw = _rng(seed, cfg, variant, layer, op, ROLE_SW).uniform(0.001, 0.01, size=n_out).astype(np.float32)
    b = _rng(seed, cfg, variant, layer, op, ROLE_B).normal(0.0, 0.02, size=n_out).astype(np.float32)
    return {"w": w, "sw": sw, "b": b, "keep": keep}


def make_x(m: int, k_in: int, *, seed: int = 0, cfg: int = 0, variant: int = 0, layer: int = 0,
           op: int = 0) -> np.ndarray:
    """Seeded int8 activations ``[m, k_in]``, uniform integers in [-127, 127]."""
    return _rng(seed, cfg, variant, layer, op, ROLE_X).integers(-127, 128, size=(m, k_in), dtype=np.int8)


def random_block_sparse(n_out: int, k_in: int, density: float, rng) -> np.ndarray:
    """Small helper for tests: int8 W with Bernoulli(density) 4x1 blocks."""
    keep = rng.random((n_out // 4, k_in)) < density
    w = rng.integers(-127, 128, size=(n_out, k_in), dtype=np.int8)
    return w * np.repeat(keep, 4, axis=0).astype(np.int8)


# ----------------------------------------------------------------------------
# workload descriptions
# ----------------------------------------------------------------------------

@dataclass(frozen=True)
class Op:
    """One sparse linear in a workload.

    ``src`` is ``"seeded"`` (input drawn with role 4 for this op) or the name of
    an earlier op of the same layer / the previous layer whose int8 output is
    this op's input (its calibrated out_scale becomes this op's x_scale).
    """
    name: str
    op_id: int
    n_out: int
    k_in: int
    sparsity: float
    kind: str
    src: str = "seeded"


@dataclass(frozen=True)
class Workload:
    name: str
    cfg: int
    variant: int
    m: int
    layers: int
    ops: Tuple[Op, ...]
    # per layer, the kind of the last op may differ (i8 feeding the next layer)
    last_layer_kinds: Optional[Dict[str, str]] = None
    notes: str = ""

    def op_kind(self, layer: int, op: Op) -> str:
        if self.last_layer_kinds and layer == self.layers - 1 and op.name in self.last_layer_kinds:
            return self.last_layer_kinds[op.name]
        return op.kind

    def op_src(self, layer: int, op: Op) -> str:
        """Source of an op's input: 'seeded', 'L<layer>.<op>'."""
        if op.src == "seeded":
            return "seeded"
        if op.src.startswith("prev:"):
            return "seeded" if layer == 0 else f"L{layer - 1}.{op.src[5:]}"
        return f"L{layer}.{op.src}"


def _distilbert_ops(sparsity: float, chained_qkv: bool = False) -> Tuple[Op, ...]:
    return (
        Op("qkv", 0, 2304, 768, sparsity, "i8", "prev:ffn2" if chained_qkv else "seeded"),
        Op("attn_out", 1, 768, 768, sparsity, "i8", "seeded"),
        Op("ffn1", 2, 3072, 768, sparsity, "i8_gelu", "attn_out"),
        Op("ffn2", 3, 768, 3072, sparsity, "i8" if chained_qkv else "f32", "ffn1"),
    )


def workloads() -> Dict[str, Workload]:
    """All workloads, keyed by name.

    c0  single linear 768x768, 80 %, M=128, fp32 out
    c1  DistilBERT FFN pair, 90 %, M=4096 (batch 32 x seq 128)
    c2  the four linears of one DistilBERT layer, 80 %, M=4096
    c3  6 stacked layers at batch 1, seq 128 / 384, sparsity 70 / 80 / 90 %
    c4  M=49152 (batch 128 x seq 384): DistilBERT layer linears at 90 % and a
        BERT-large FFN pair at 80 %
    """
    w: Dict[str, Workload] = {}
    w["c0"] = Workload("c0", 0, 0, 128, 1, (Op("linear", 0, 768, 768, 0.8, "f32"),),
                       notes="single sparse linear 768x768, 80%, batch 1 x seq 128")
    w["c1"] = Workload("c1", 1, 0, 4096, 1, (
        Op("ffn1", 2, 3072, 768, 0.9, "i8_gelu"),
        Op("ffn2", 3, 768, 3072, 0.9, "f32", "ffn1"),
    ), notes="DistilBERT FFN pair, 90%, batch 32 x seq 128")
    w["c2"] = Workload("c2", 2, 0, 4096, 1, _distilbert_ops(0.8),
                       notes="one DistilBERT layer's linears, 80%, batch 32 x seq 128")
    v = 0
    for seq in (128, 384):
        for s in (0.7, 0.8, 0.9):
            name = f"c3_seq{seq}_s{int(round(s * 100))}"
            w[name] = Workload(name, 3, v, seq, 6, _distilbert_ops(s, chained_qkv=True),
                               last_layer_kinds={"ffn2": "f32"},
                               notes=f"6 DistilBERT layers, batch 1 x seq {seq}, {int(round(s*100))}%")
            v += 1
    w["c4"] = Workload("c4", 4, 0, 49152, 1, _distilbert_ops(0.9),
                       notes="DistilBERT layer linears, 90%, batch 128 x seq 384")
    w["c4_bertl"] = Workload("c4_bertl", 4, 1, 49152, 1, (
        Op("ffn1", 2, 4096, 1024, 0.8, "i8_gelu"),
        Op("ffn2", 3, 1024, 4096, 0.8, "f32", "ffn1"),
    ), notes="BERT-large FFN pair, 80%, batch 128 x seq 384")
    return w


def op_weight(wl: Workload, layer: int, op: Op, seed: int = 0) -> Dict[str, np.ndarray]:
    return make_weight(op.n_out, op.k_in, op.sparsity, seed=seed, cfg=wl.cfg,
                       variant=wl.variant, layer=layer, op=op.op_id)


def op_seeded_x(wl: Workload, layer: int, op: Op, m: Optional[int] = None, seed: int = 0) -> np.ndarray:
    return make_x(wl.m if m is None else m, op.k_in, seed=seed, cfg=wl.cfg, variant=wl.variant,
                  layer=layer, op=op.op_id)


def op_list(wl: Workload) -> List[Tuple[int, Op]]:
    """(layer, op) pairs in execution order."""
    return [(layer, op) for layer in range(wl.layers) for op in wl.ops]
