"""Plain fp64 oracle of the LoRA linear forward and backward -- TEST INFRASTRUCTURE.

Not part of the product path; see the package docstring for who may call it.
All arrays are row-major numpy arrays.  Inputs arrive as bfloat16 bit patterns
(uint16) and are decoded exactly to float64 here; every product below is a
float64 numpy matmul.
"""
from __future__ import annotations

from typing import Optional, Sequence, Tuple

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact decode of bfloat16 bit patterns: the 16 bits are the top half of a float32."""
    u32 = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u32.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (nearest, ties to even) for bit-exact checks.

    Goes through float32 first; that double rounding is harmless for the
    small-integer values this is used on."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def f64_to_bf16_rne(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 bit patterns, nearest with ties to even,
    in one rounding step (no intermediate float32).

    A finite x = m 2^e with 0.5 <= |m| < 1 has bfloat16 neighbours spaced
    2^(e-8) apart (8 significant bits); below the smallest normal (2^-126) the
    spacing stays 2^-133.  x / spacing is an exact power-of-two scaling, so
    rounding it to an integer with ties to even (numpy.rint) and scaling back
    gives the bfloat16 value exactly; that value is exact in float32, whose top
    16 bits are the pattern.  NaN and infinity are not handled (the data here
    has none)."""
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    e = np.maximum(e, -125)
    q = np.ldexp(1.0, e - 8)
    y = np.rint(x / q) * q
    return (y.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)


def lora_scale(alpha: float, r: int) -> float:
    """LoRA scale s = alpha / r.  The paper's Eq. 1 shows no scale; its config
    (Listing 3) carries LORA_ALPHA and LORA_R, whose defaults (16, 16) give s = 1,
    which is Eq. 1 as printed."""
    return float(alpha) / float(r)


def _f64(a: np.ndarray) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return bf16_bits_to_f64(a)
    return a.astype(np.float64, copy=False)


def lora_rank_activation(X, A) -> np.ndarray:
    """The rank-r activation U = X A^T of Eq. 1 (the A x term, row-major), [m, r]."""
    return _f64(X) @ _f64(A).T


def lora_forward(X, W, A, B, alpha: float) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. 1 (Section 3): U = X A^T; Y = X W^T + s U B^T, with b0 = 0.

    X [m,k], W [n,k] (frozen W0, stored out x in), A [r,k], B [n,r].
    Returns (U [m,r], Y [m,n]) in float64."""
    X, W, A, B = _f64(X), _f64(W), _f64(A), _f64(B)
    s = lora_scale(alpha, A.shape[0])
    U = X @ A.T
    Y = X @ W.T + s * (U @ B.T)
    return U, Y


def lora_backward(dY, X, W, A, B, alpha: float
                  ) -> Tuple[np.ndarray, np.ndarray, np.ndarray, np.ndarray]:
    """Chain rule through Eq. 1 for the trainable A and B (W0 frozen: no dW).

    Returns (dU [m,r], dX [m,k], dA [r,k], dB [n,r]) in float64, where
    dU = s dY B is the gradient of the rank-r activation U = X A^T."""
    dY, X, W, A, B = _f64(dY), _f64(X), _f64(W), _f64(A), _f64(B)
    s = lora_scale(alpha, A.shape[0])
    U = X @ A.T
    dU = s * (dY @ B)
    dX = dY @ W + dU @ A
    dB = s * (dY.T @ U)
    dA = dU.T @ X
    return dU, dX, dA, dB


def lora_merged_weight(W, A, B, alpha: float, sign: int = 1) -> np.ndarray:
    """The merged weight of Eq. 1's second form, W0 x + B A x = (W0 + B A) x,
    with the LoRA scale: W + sign s B A (sign = -1 unmerges).  [n, k], float64."""
    W, A, B = _f64(W), _f64(A), _f64(B)
    s = lora_scale(alpha, A.shape[0])
    return W + float(sign) * s * (B @ A)


def lora_merge_bf16(W, A, B, alpha: float, sign: int = 1) -> np.ndarray:
    """lora_merged_weight rounded once to bfloat16 (nearest-even): the stored
    result of a merge or unmerge.  Returns uint16 bit patterns [n, k]."""
    return f64_to_bf16_rne(lora_merged_weight(W, A, B, alpha, sign))


def dropout_keep(keep_bits, k: int) -> np.ndarray:
    """Decode a packed keep mask ([m, k/8] bytes, bit l % 8 of byte l // 8 of
    row i keeps element (i, l)) into a float64 0/1 matrix [m, k]."""
    b = np.asarray(keep_bits, dtype=np.uint8)
    return np.unpackbits(b, axis=1, bitorder="little")[:, :k].astype(np.float64)


def dropped_input(X, keep_bits, p: float) -> np.ndarray:
    """The adapter's input under LoRA dropout (Listing 3's LORA_DROPOUT; the
    dropout acts on the input of A only, the frozen W0 sees x unchanged):
    D = keep * X / (1 - p), the usual inverted-dropout scaling during training."""
    X = _f64(X)
    return dropout_keep(keep_bits, X.shape[1]) * X / (1.0 - float(p))


def lora_forward_dropout(X, W, A, B, keep_bits, p: float, alpha: float
                         ) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. 1 with dropout on the adapter input: U = D A^T, Y = X W^T + s U B^T,
    D = dropped_input(X).  Returns (U [m,r], Y [m,n]) in float64."""
    X, W, A, B = _f64(X), _f64(W), _f64(A), _f64(B)
    s = lora_scale(alpha, A.shape[0])
    D = dropped_input(X, keep_bits, p)
    U = D @ A.T
    Y = X @ W.T + s * (U @ B.T)
    return U, Y


def lora_backward_dropout(dY, X, W, A, B, keep_bits, p: float, alpha: float
                          ) -> Tuple[np.ndarray, np.ndarray, np.ndarray, np.ndarray]:
    """Chain rule through lora_forward_dropout for a fixed mask: with
    dU = s dY B,  dX = dY W + keep * (dU A) / (1 - p),  dB = s dY^T U,
    dA = dU^T D.  Returns (dU, dX, dA, dB) in float64."""
    dY, X, W, A, B = _f64(dY), _f64(X), _f64(W), _f64(A), _f64(B)
    s = lora_scale(alpha, A.shape[0])
    keep = dropout_keep(keep_bits, X.shape[1])
    D = keep * X / (1.0 - float(p))
    U = D @ A.T
    dU = s * (dY @ B)
    dX = dY @ W + keep * (dU @ A) / (1.0 - float(p))
    dB = s * (dY.T @ U)
    dA = dU.T @ D
    return dU, dX, dA, dB


def lora_forward_rows(X, W, A, B, alpha: float, rows: Sequence[int]
                      ) -> Tuple[np.ndarray, np.ndarray]:
    """The forward restricted to the token rows `rows` (each output row of Eq. 1
    depends only on the same row of X).  Returns (U[rows], Y[rows])."""
    idx = np.asarray(rows, dtype=np.int64)
    return lora_forward(np.asarray(X)[idx], W, A, B, alpha)


def lora_backward_rows(dY, X, W, A, B, alpha: float, rows: Optional[Sequence[int]]
                       ) -> Tuple[np.ndarray, np.ndarray, np.ndarray, np.ndarray]:
    """Backward with dX evaluated only at token rows `rows` (dX row i depends only
    on row i of dY).  dU, dA and dB reduce over all tokens and are returned whole.

    Returns (dU [m,r], dX[rows] [len(rows),k], dA [r,k], dB [n,r])."""
    dY64, X64, W64, A64, B64 = _f64(dY), _f64(X), _f64(W), _f64(A), _f64(B)
    s = lora_scale(alpha, A64.shape[0])
    U = X64 @ A64.T
    dU = s * (dY64 @ B64)
    idx = np.arange(dY64.shape[0]) if rows is None else np.asarray(rows, dtype=np.int64)
    dX = dY64[idx] @ W64 + dU[idx] @ A64
    dB = s * (dY64.T @ U)
    dA = dU.T @ X64
    return dU, dX, dA, dB


def lora_group_forward(X, Ws: Sequence, As: Sequence, Bs: Sequence, alpha: float
                       ) -> Tuple[list, list]:
    """G adapted projections that read one input X (the query, key and value
    projections of an attention block; Section 3 adapts the query and value
    projections): for each g, Eq. 1 with its own W_g, A_g, B_g and the shared
    rank and alpha.  Returns ([U_g], [Y_g]) in float64."""
    X = _f64(X)
    outs = [lora_forward(X, W, A, B, alpha) for W, A, B in zip(Ws, As, Bs)]
    return [u for u, _ in outs], [y for _, y in outs]


def lora_group_backward(dYs: Sequence, X, Ws: Sequence, As: Sequence, Bs: Sequence, alpha: float,
                        rows: Optional[Sequence[int]] = None) -> Tuple[list, np.ndarray, list, list]:
    """Chain rule through lora_group_forward.  X feeds every projection, so its
    gradient is the sum of the projections' contributions:
        dX = sum_g (dY_g W_g + dU_g A_g),   dU_g = s dY_g B_g,
        dB_g = s dY_g^T U_g,   dA_g = dU_g^T X.
    With `rows`, dX is evaluated only at those token rows.  Returns
    ([dU_g], dX, [dA_g], [dB_g]) in float64."""
    X = _f64(X)
    idx = np.arange(X.shape[0]) if rows is None else np.asarray(rows, dtype=np.int64)
    dUs, dAs, dBs = [], [], []
    dX = np.zeros((len(idx), X.shape[1]))
    for dY, W, A, B in zip(dYs, Ws, As, Bs):
        dU, dXg, dA, dB = lora_backward_rows(dY, X, W, A, B, alpha, idx)
        dUs.append(dU)
        dAs.append(dA)
        dBs.append(dB)
        dX = dX + dXg
    return dUs, dX, dAs, dBs
