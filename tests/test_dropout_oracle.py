"""Pins of the oracle's LoRA dropout (Listing 3's LORA_DROPOUT on the adapter
input: D = keep * X / (1 - p), U = D A^T, Y = X W^T + s U B^T).

  * p0         -- p = 0 with every element kept is the plain method, exactly.
  * drop_all   -- nothing kept: U = 0, Y = X W^T, dA = dB = 0, dX = dY W, exactly.
  * same_route -- the LoRA branch equals the plain oracle run on the dropped
                  input D (a different route through the code), and the frozen
                  path still sees X.
  * fd         -- central finite differences of L = <dY, Y> in entries of X, A
                  and B for a fixed mask (L is affine in each entry, so the
                  quotient is exact up to rounding).
  * brute      -- scalar loops over the index definitions with an explicit
                  per-element mask, tiny shapes.
  * bits       -- the packed mask layout: bit l % 8 of byte l // 8 of row i.
A last test plants plausible mistakes and checks each is caught.
"""
import numpy as np
import pytest

import oracle
from lora_synth import Shape, gen_inputs, gen_keep_mask


def _case(m, n, k, r, alpha, p, seed):
    t = gen_inputs(Shape("pin", m, n, k, r, alpha, seed), seed=seed, b_std=0.3)
    t["keep"] = gen_keep_mask(m, k, p, seed + 100)
    return t


def _o_fwd(t, p, alpha):
    return oracle.lora_forward_dropout(t["X"], t["W"], t["A"], t["B"], t["keep"], p, alpha)


def _o_bwd(t, p, alpha):
    return oracle.lora_backward_dropout(t["dY"], t["X"], t["W"], t["A"], t["B"], t["keep"], p, alpha)


def check_p0(fwd, bwd):
    t = _case(12, 16, 24, 4, 8.0, 0.0, 1)
    t["keep"][:] = 0xFF
    U, Y = fwd(t, 0.0, 8.0)
    U0, Y0 = oracle.lora_forward(t["X"], t["W"], t["A"], t["B"], 8.0)
    g = bwd(t, 0.0, 8.0)
    g0 = oracle.lora_backward(t["dY"], t["X"], t["W"], t["A"], t["B"], 8.0)
    return (np.array_equal(U, U0) and np.array_equal(Y, Y0)
            and all(np.array_equal(a, b) for a, b in zip(g, g0)))


def check_drop_all(fwd, bwd):
    t = _case(10, 24, 16, 3, 6.0, 0.3, 2)
    t["keep"][:] = 0
    U, Y = fwd(t, 0.3, 6.0)
    dU, dX, dA, dB = bwd(t, 0.3, 6.0)
    X, W, dY = (oracle.bf16_bits_to_f64(t[x]) for x in ("X", "W", "dY"))
    return (not U.any() and np.array_equal(Y, X @ W.T) and not dA.any() and not dB.any()
            and np.array_equal(dX, dY @ W))


def check_same_route(fwd, bwd):
    p, alpha = 0.25, 16.0
    t = _case(9, 32, 40, 8, alpha, p, 3)
    D = oracle.dropped_input(t["X"], t["keep"], p)
    U, Y = fwd(t, p, alpha)
    Ud, Yd = oracle.lora_forward(D, t["W"], t["A"], t["B"], alpha)   # plain method on the dropped input
    X, W = oracle.bf16_bits_to_f64(t["X"]), oracle.bf16_bits_to_f64(t["W"])
    ok = np.allclose(U, Ud, rtol=0, atol=1e-12) and np.allclose(Y - X @ W.T, Yd - D @ W.T, rtol=0, atol=1e-12)
    dU, dX, dA, dB = bwd(t, p, alpha)
    dUd, dXd, dAd, dBd = oracle.lora_backward(t["dY"], D, t["W"], t["A"], t["B"], alpha)
    dY = oracle.bf16_bits_to_f64(t["dY"])
    keep = oracle.dropout_keep(t["keep"], X.shape[1])
    # the plain backward on D gives dD = dY W + dU A; the LoRA part of dX is keep / (1-p) times its second term
    ok = ok and np.allclose(dA, dAd, rtol=0, atol=1e-12) and np.allclose(dB, dBd, rtol=0, atol=1e-12)
    ok = ok and np.allclose(dX - dY @ W, keep * (dXd - dY @ W) / (1 - p), rtol=0, atol=1e-12)
    return bool(ok)


def check_fd(fwd, bwd):
    p, alpha = 0.4, 4.0
    t = _case(5, 6, 8, 2, alpha, p, 4)
    dY = oracle.bf16_bits_to_f64(t["dY"])
    _, dX, dA, dB = bwd(t, p, alpha)
    f = {x: oracle.bf16_bits_to_f64(t[x]) for x in ("X", "A", "B")}

    def L(vals):
        tt = dict(t)
        tt.update(vals)
        return float(np.sum(dY * fwd(tt, p, alpha)[1]))

    h = 2.0 ** -10
    rng = np.random.default_rng(5)
    for name, grad in (("X", dX), ("A", dA), ("B", dB)):
        for _ in range(6):
            idx = tuple(rng.integers(0, s) for s in f[name].shape)
            plus, minus = f[name].copy(), f[name].copy()
            plus[idx] += h
            minus[idx] -= h
            fd = (L({name: plus}) - L({name: minus})) / (2 * h)
            if abs(fd - grad[idx]) > 1e-9 * max(1.0, abs(grad[idx])):
                return False
    return True


def check_brute(fwd, bwd):
    p, alpha = 0.5, 3.0
    t = _case(3, 4, 8, 2, alpha, p, 6)
    X, W, A, B, dY = (oracle.bf16_bits_to_f64(t[x]) for x in ("X", "W", "A", "B", "dY"))
    m, k = X.shape
    n, r = W.shape[0], A.shape[0]
    s = alpha / r
    kp = [[(int(t["keep"][i, l // 8]) >> (l % 8)) & 1 for l in range(k)] for i in range(m)]
    U = [[sum(kp[i][l] * X[i, l] / (1 - p) * A[q, l] for l in range(k)) for q in range(r)] for i in range(m)]
    Y = [[sum(X[i, l] * W[j, l] for l in range(k)) + s * sum(U[i][q] * B[j, q] for q in range(r))
          for j in range(n)] for i in range(m)]
    dU = [[s * sum(dY[i, j] * B[j, q] for j in range(n)) for q in range(r)] for i in range(m)]
    dX = [[sum(dY[i, j] * W[j, l] for j in range(n))
           + kp[i][l] / (1 - p) * sum(dU[i][q] * A[q, l] for q in range(r)) for l in range(k)] for i in range(m)]
    dA = [[sum(dU[i][q] * kp[i][l] * X[i, l] / (1 - p) for i in range(m)) for l in range(k)] for q in range(r)]
    dB = [[s * sum(dY[i, j] * U[i][q] for i in range(m)) for q in range(r)] for j in range(n)]
    Uo, Yo = fwd(t, p, alpha)
    _, dXo, dAo, dBo = bwd(t, p, alpha)
    return all(np.allclose(a, np.array(b), rtol=0, atol=1e-12)
               for a, b in ((Uo, U), (Yo, Y), (dXo, dX), (dAo, dA), (dBo, dB)))


def check_bits(fwd, bwd):
    keep = np.array([[0b00000101, 0b10000000]], dtype=np.uint8)
    ref = np.zeros((1, 16))
    ref[0, [0, 2, 15]] = 1.0
    return bool(np.array_equal(oracle.dropout_keep(keep, 16), ref))


CHECKS = [check_p0, check_drop_all, check_same_route, check_fd, check_brute, check_bits]


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_dropout_pin(check):
    assert check(_o_fwd, _o_bwd)


def test_keep_mask_density():
    keep = gen_keep_mask(256, 512, 0.05, 7)
    frac = oracle.dropout_keep(keep, 512).mean()
    assert abs(frac - 0.95) < 0.005


# ---- planted mistakes (each must fail at least one pin) ---------------------
def _parts(t, p):
    X, W, A, B, dY = (oracle.bf16_bits_to_f64(t[x]) for x in ("X", "W", "A", "B", "dY"))
    keep = oracle.dropout_keep(t["keep"], X.shape[1])
    return X, W, A, B, dY, keep


def _mut_mask_on_frozen_path(t, p, alpha):
    X, W, A, B, dY, keep = _parts(t, p)
    D = keep * X / (1 - p)
    s = alpha / A.shape[0]
    U = D @ A.T
    return U, D @ W.T + s * U @ B.T


def _mut_no_rescale(t, p, alpha):
    X, W, A, B, dY, keep = _parts(t, p)
    s = alpha / A.shape[0]
    U = (keep * X) @ A.T
    return U, X @ W.T + s * U @ B.T


def _mut_bwd_dx_unmasked(t, p, alpha):
    dU, dX, dA, dB = _o_bwd(t, p, alpha)
    X, W, A, B, dY, keep = _parts(t, p)
    return dU, dY @ W + dU @ A / (1 - p), dA, dB


def _mut_bwd_da_unmasked(t, p, alpha):
    dU, dX, dA, dB = _o_bwd(t, p, alpha)
    X, W, A, B, dY, keep = _parts(t, p)
    return dU, dX, dU.T @ X / (1 - p), dB


def _mut_bits_reversed(t, p, alpha):
    tt = dict(t)
    tt["keep"] = np.packbits(np.unpackbits(t["keep"], axis=1, bitorder="little"), axis=1, bitorder="big")
    return _o_fwd(tt, p, alpha)


MUTANTS = [("mask_on_frozen_path", _mut_mask_on_frozen_path, _o_bwd),
           ("no_rescale", _mut_no_rescale, _o_bwd),
           ("dx_unmasked", _o_fwd, _mut_bwd_dx_unmasked),
           ("da_unmasked", _o_fwd, _mut_bwd_da_unmasked),
           ("bits_reversed", _mut_bits_reversed, _o_bwd)]


@pytest.mark.parametrize("name,fwd,bwd", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_dropout_mistake(name, fwd, bwd):
    assert not all(check(fwd, bwd) for check in CHECKS)
