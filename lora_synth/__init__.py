"""Seeded synthetic inputs for the LoRA-adapted linear layer.

This module is shared by the fp64 oracle and the HIP path and therefore holds
none of the method's arithmetic: it only names the workload shapes and draws
seeded random tensors, rounded once to bfloat16 bit patterns.  Both sides
receive the same bits.

Shapes follow the Llama-2 projection sizes the paper fine-tunes (Section 3,
"Model Transfer API": LoRA on the attention projections of a Llama-2 decoder;
Section 4 uses bf16 parameters).  The token count m = batch x sequence stands
for long retrieval-augmented prompts; tokens are dense (no padding, no masks).

Distributions (one reading, recorded with every result):
  X  ~ N(0, 1)              layer input, [m, k]
  W  ~ N(0, std 1/sqrt(k))  frozen weight, [n, k]   (variance 1/k)
  A  ~ U(-1/sqrt(k), +1/sqrt(k))  LoRA down, [r, k]
  B  ~ N(0, std 0.02)       LoRA up, [n, r]
  dY ~ N(0, 1)              upstream gradient, [m, n]
Each tensor is drawn as float32 from numpy's PCG64 generator in the fixed
order X, W, A, B, dY, then rounded to bfloat16 with round-to-nearest-even.
Seed = 1000 * config_index + projection_index.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

__all__ = [
    "Shape", "CONFIGS", "config_shapes", "round_to_bf16_bits", "bf16_bits_to_f32",
    "gen_inputs", "gen_ternary_inputs", "gen_keep_mask", "LAYER_GROUPS", "gen_group_inputs",
]


@dataclasses.dataclass(frozen=True)
class Shape:
    """One LoRA-linear problem: Y[m,n] = X[m,k] W[n,k]^T + (alpha/r) (X A^T) B^T."""
    name: str
    m: int
    n: int
    k: int
    r: int
    alpha: float
    seed: int

    @property
    def flops_fwd_bwd(self) -> int:
        """Algorithmic flops of forward + backward: 4mnk + 6mr(n+k)."""
        m, n, k, r = self.m, self.n, self.k, self.r
        return 4 * m * n * k + 6 * m * r * (n + k)


def _cfg(ci: int, name: str, m, n, k, r, alpha, proj: int = 0) -> Shape:
    return Shape(name, m, n, k, r, float(alpha), 1000 * ci + proj)


# Llama-2-13B decoder layer projections (hidden 5120, MLP 13824), in layer order.
_L13 = [("q_proj", 5120, 5120), ("k_proj", 5120, 5120), ("v_proj", 5120, 5120),
        ("o_proj", 5120, 5120), ("gate_proj", 13824, 5120), ("up_proj", 13824, 5120),
        ("down_proj", 5120, 13824)]

CONFIGS: Dict[str, List[Shape]] = {
    "tiny": [_cfg(0, "tiny", 256, 512, 512, 8, 16)],
    "llama2_7b_q_proj": [_cfg(1, "llama2_7b_q_proj", 2048, 4096, 4096, 8, 16)],
    "llama2_7b_up_proj": [_cfg(2, "llama2_7b_up_proj", 4096, 11008, 4096, 16, 32)],
    "llama2_7b_down_proj": [_cfg(3, "llama2_7b_down_proj", 8192, 4096, 11008, 64, 128)],
    "llama2_13b_layer": [_cfg(4, f"llama2_13b_{p}", 4096, n, k, 8, 16, proj=i)
                         for i, (p, n, k) in enumerate(_L13)],
}
# The three Llama-2-7B projection shapes above as one step (q_proj, up_proj,
# down_proj back to back), each with its own configuration's seed.
CONFIGS["llama2_7b_shapes"] = (CONFIGS["llama2_7b_q_proj"] + CONFIGS["llama2_7b_up_proj"]
                               + CONFIGS["llama2_7b_down_proj"])
CONFIG_ORDER = ["tiny", "llama2_7b_q_proj", "llama2_7b_up_proj", "llama2_7b_down_proj",
                "llama2_13b_layer"]


def config_shapes(name: str) -> List[Shape]:
    return CONFIGS[name]


def round_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest, ties to even.

    The inputs here are finite; NaN/Inf are not produced by the generators."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float32 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def gen_inputs(shape: Shape, seed: Optional[int] = None, b_std: float = 0.02,
               zero_a: bool = False, zero_b: bool = False) -> Dict[str, np.ndarray]:
    """Draw X, W, A, B, dY for `shape` as bf16 bit arrays (uint16, row-major).

    `b_std` overrides B's standard deviation (a large B makes the LoRA branch a
    large share of Y).  `zero_a` / `zero_b` replace A or B by zeros after the
    draw, so the other tensors are unchanged (B = 0 is the paper's LoRA
    initialisation)."""
    m, n, k, r = shape.m, shape.n, shape.k, shape.r
    rng = np.random.default_rng(shape.seed if seed is None else seed)
    inv = 1.0 / np.sqrt(k)
    X = rng.standard_normal((m, k), dtype=np.float32)
    W = (rng.standard_normal((n, k), dtype=np.float32) * np.float32(inv))
    A = rng.uniform(-inv, inv, size=(r, k)).astype(np.float32)
    B = (rng.standard_normal((n, r), dtype=np.float32) * np.float32(b_std))
    dY = rng.standard_normal((m, n), dtype=np.float32)
    out = {name: round_to_bf16_bits(v) for name, v in
           (("X", X), ("W", W), ("A", A), ("B", B), ("dY", dY))}
    if zero_a:
        out["A"][:] = 0
    if zero_b:
        out["B"][:] = 0
    return out


def gen_ternary_inputs(m: int, n: int, k: int, r: int, seed: int,
                       density: float = 0.02) -> Dict[str, np.ndarray]:
    """Sparse {-1, 0, +1} tensors as bf16 bits.

    With few non-zeros per row every partial sum is a small integer, so any
    summation order in fp32 is exact; used for bit-exact tiling checks."""
    rng = np.random.default_rng(seed)

    def tern(shape, d):
        v = rng.random(shape) < d
        s = np.where(rng.random(shape) < 0.5, -1.0, 1.0)
        return round_to_bf16_bits((v * s).astype(np.float32))

    return {"X": tern((m, k), density), "W": tern((n, k), density),
            "A": tern((r, k), density), "B": tern((n, r), 4 * density),
            "dY": tern((m, n), density)}


def gen_keep_mask(m: int, k: int, p: float, seed: int) -> np.ndarray:
    """Seeded dropout keep mask for the adapter input, packed as the library
    takes it: [m, k / 8] bytes, bit (l % 8) of byte l // 8 of row i set when
    element (i, l) is kept.  Each element is kept independently with
    probability 1 - p (numpy PCG64, float64 uniforms compared with p)."""
    assert k % 8 == 0
    rng = np.random.default_rng(seed)
    keep = rng.random((m, k)) >= p
    return np.packbits(keep, axis=1, bitorder="little")


# Projections of one decoder layer that read the same input: q, k, v (the
# attention input) and gate, up (the MLP input); o and down stand alone.
LAYER_GROUPS: Dict[str, List[List[int]]] = {"llama2_13b_layer": [[0, 1, 2], [3], [4, 5], [6]]}


def gen_group_inputs(shapes: List[Shape], b_std: float = 0.02) -> Dict[str, object]:
    """Inputs of projections that share one layer input: X is the first
    projection's draw; W, A, B and dY of each projection come from its own
    seeded draw (gen_inputs), so they equal the per-projection inputs.
    Returns {"X": X, "W": [..], "A": [..], "B": [..], "dY": [..]}."""
    s0 = shapes[0]
    assert all(s.m == s0.m and s.k == s0.k and s.r == s0.r and s.alpha == s0.alpha for s in shapes)
    per = [gen_inputs(s, b_std=b_std) for s in shapes]
    return {"X": per[0]["X"], "W": [t["W"] for t in per], "A": [t["A"] for t in per],
            "B": [t["B"] for t in per], "dY": [t["dY"] for t in per]}
