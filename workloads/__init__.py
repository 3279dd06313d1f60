"""Seeded synthetic workloads for the protected attention layer.

This module is shared by the CPU oracle, the tests and the benchmark. It
holds shapes, seeds and random draws only: no checksum, GEMM, softmax or
correction arithmetic lives here. Inputs are returned as float32 NumPy
arrays whose values are already representable in the storage dtype, so the
oracle and the GPU path see bit-identical operands.

Layer convention (paper Sec. 2.1, Eq. 1-2; GPT-2 style packed weights):
    X    [B, S, H]          activations, token-major
    Wqkv [H, 3H]            Q = X Wqkv[:, 0:H], K = ..[:, H:2H], V = ..[:, 2H:3H]
    Wo   [H, H]             O = CL Wo
    dO   [B, S, H]          upstream gradient
Head h owns columns [h*d, (h+1)*d) of Q, K, V and CL.
"""
from __future__ import annotations

import dataclasses
import numpy as np

# Op tags of the protected GEMM outputs (paper Table 1 notation; the
# backward ops extend it). Faults and events name their op by these strings.
FWD_OPS = ("Q", "K", "V", "AS", "CL", "O")
BWD_OPS = ("dCL", "dWO", "dAP", "dV", "dQ", "dK", "dWQ", "dWK", "dWV", "dX")
ALL_OPS = FWD_OPS + BWD_OPS


@dataclasses.dataclass(frozen=True)
class LayerShape:
    """Shape and value recipe of one attention-layer workload."""
    name: str
    batch: int
    seq: int
    hidden: int
    heads: int
    causal: bool
    dtype: str            # storage dtype: "bf16" or "f32"
    w_std: float          # std of Wqkv / Wo entries
    backward: bool        # whether the workload includes the backward chain
    block_rows: int = 128  # checksum block R along token axes

    @property
    def head_dim(self) -> int:
        return self.hidden // self.heads

    @property
    def tokens(self) -> int:
        return self.batch * self.seq


# The five workloads: shapes of the paper's model families (BERT-base /
# GPT-2 small encoder and decoder layers, and two larger decoder layers).
C1 = LayerShape("single-head-fp32-S128-H64", 1, 128, 64, 1, False, "f32", 0.02, False)
C2 = LayerShape("encoder-B8-S512-H768-12x64", 8, 512, 768, 12, False, "bf16", 0.02, True)
C3 = LayerShape("gpt2-causal-B8-S1024-H768-12x64", 8, 1024, 768, 12, True, "bf16", 0.02, True)
C4 = LayerShape("decoder-causal-B4-S2048-H4096-32x128", 4, 2048, 4096, 32, True, "bf16", 0.01, True)
C5 = LayerShape("stress-causal-B1-S4096-H5120-40x128", 1, 4096, 5120, 40, True, "bf16", 0.01, True)
CONFIGS = {"c1": C1, "c2": C2, "c3": C3, "c4": C4, "c5": C5}
CONFIG_INDEX = {"c1": 1, "c2": 2, "c3": 3, "c4": 4, "c5": 5}


def data_seed(cfg_key: str) -> int:
    return 1000 + CONFIG_INDEX[cfg_key]


def fault_seed(cfg_key: str, step: int) -> int:
    return 2000 + CONFIG_INDEX[cfg_key] * 1000 + step


def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    """Round a float array to the storage dtype (round-to-nearest-even),
    returned as float32. Uses torch's conversion; inputs only."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "f32":
        return a
    if dtype == "bf16":
        import torch
        return torch.from_numpy(a).to(torch.bfloat16).to(torch.float32).numpy()
    raise ValueError(f"unknown storage dtype {dtype!r}")


def make_shape(batch, seq, hidden, heads, *, causal=False, dtype="bf16",
               w_std=0.02, backward=True, block_rows=None, name=None) -> LayerShape:
    """A custom workload shape (tests use small ones with several tiles and
    ragged edges)."""
    if block_rows is None:
        block_rows = min(128, seq)
    return LayerShape(name or f"custom-B{batch}-S{seq}-H{hidden}-{heads}h",
                      batch, seq, hidden, heads, causal, dtype, w_std, backward,
                      block_rows)


def make_inputs(shape: LayerShape, seed: int) -> dict:
    """X ~ N(0,1), Wqkv, Wo ~ N(0, w_std^2), dO ~ N(0,1), drawn from PCG64(seed)
    in that order and rounded to the storage dtype."""
    rng = np.random.Generator(np.random.PCG64(seed))
    B, S, H = shape.batch, shape.seq, shape.hidden
    X = rng.standard_normal((B, S, H), dtype=np.float32)
    Wqkv = rng.standard_normal((H, 3 * H), dtype=np.float32) * np.float32(shape.w_std)
    Wo = rng.standard_normal((H, H), dtype=np.float32) * np.float32(shape.w_std)
    dO = rng.standard_normal((B, S, H), dtype=np.float32)
    return {k: to_storage(v, shape.dtype) for k, v in
            dict(X=X, Wqkv=Wqkv, Wo=Wo, dO=dO).items()}


@dataclasses.dataclass(frozen=True)
class Fault:
    """One injected fault in element (row, col) of op's output for batch b
    and head h, after the output is rounded to storage: mode "set"
    overwrites it with value (rounded to storage), mode "flip" flips the
    most significant exponent bit of the stored value (value unused)."""
    op: str
    b: int
    h: int
    row: int
    col: int
    value: float
    mode: str = "set"

    def as_tuple(self):
        t = (self.op, self.b, self.h, self.row, self.col, self.value)
        return t if self.mode == "set" else t + (self.mode,)


def op_extent(shape: LayerShape, op: str):
    """(n_b, n_h, rows, cols) of the index space the fault coordinates of op
    live in. Per-head ops use head-local columns; O and dX use the full
    hidden width with h = 0; weight gradients use b = h = 0."""
    B, S, H, nh, d = shape.batch, shape.seq, shape.hidden, shape.heads, shape.head_dim
    if op in ("Q", "K", "V", "CL", "dCL", "dV", "dQ", "dK"):
        return B, nh, S, d
    if op in ("AS", "dAP"):
        return B, nh, S, S
    if op in ("O", "dX"):
        return B, 1, S, H
    if op in ("dWO", "dWQ", "dWK", "dWV"):
        return 1, 1, H, H
    raise ValueError(op)


KIND_VALUES = {
    "inf": float("inf"),
    "-inf": float("-inf"),
    "nan": float("nan"),
    "+1e10": 1e10,
    "-1e10": -1e10,
    "1e6": 1e6,
    "1e10": 1e10,
    "1e30": 1e30,
    "+1e6": 1e6,
    "-1e6": -1e6,
    "+1e30": 1e30,
    "-1e30": -1e30,
}


def draw_faults(shape: LayerShape, seed: int, n: int, ops, kinds,
                distinct=True) -> list:
    """Draw n faults at uniform positions, op and kind uniform over the given
    lists. Positions of score-shaped ops (AS, dAP) are restricted to the
    unmasked part (key <= query) under a causal mask. With distinct=True no
    two faults share a row or a column of the same (op, b, h), so at most one
    fault lands in any checksum row or column vector."""
    rng = np.random.Generator(np.random.PCG64(seed))
    ops = list(ops)
    kinds = list(kinds)
    out = []
    used_rows, used_cols = set(), set()
    tries = 0
    while len(out) < n:
        tries += 1
        if tries > 100000:
            raise RuntimeError("could not place distinct faults")
        op = ops[int(rng.integers(len(ops)))]
        kind = kinds[int(rng.integers(len(kinds)))]
        nb, nhh, rows, cols = op_extent(shape, op)
        b = int(rng.integers(nb))
        h = int(rng.integers(nhh))
        r = int(rng.integers(rows))
        if op in ("AS", "dAP") and shape.causal:
            c = int(rng.integers(r + 1))
        else:
            c = int(rng.integers(cols))
        if distinct:
            kr, kc = (op, b, h, r), (op, b, h, c)
            if kr in used_rows or kc in used_cols:
                continue
            used_rows.add(kr)
            used_cols.add(kc)
        out.append(Fault(op, b, h, r, c, KIND_VALUES[kind]))
    return out
