"""Pins of the oracle's grouped projections: G adapted projections that read
one input X (Section 3 adapts the query and value projections of each
attention block; q, k and v read the same input), each with its own W_g, A_g,
B_g, and the input gradient summed over the group.

  * single   -- a group of one is the plain method, exactly.
  * stacked  -- the group equals ONE LoRA linear (another route through the
                oracle) with the weights stacked, W = [W_1; ...; W_G],
                A = [A_1; ...; A_G] of rank G r, B block-diagonal, and the same
                scale s (alpha' = s G r): Y and U split by columns, dX equal,
                dA split by rows, dB the diagonal blocks.
  * fd       -- central finite differences of L = sum_g <dY_g, Y_g> in entries
                of X (the summed input gradient), A_g and B_g.
  * brute    -- scalar loops over the index definitions, tiny shapes.
  * rows     -- the row-restricted dX equals those rows of the full dX.
A last test plants plausible mistakes and checks each is caught.
"""
import numpy as np
import pytest

import oracle
from lora_synth import Shape, gen_group_inputs


def _group(ns, m, k, r, alpha, seed, b_std=0.3):
    shapes = [Shape(f"g{i}", m, n, k, r, alpha, seed + i) for i, n in enumerate(ns)]
    return gen_group_inputs(shapes, b_std=b_std)


def _fwd(t, alpha):
    return oracle.lora_group_forward(t["X"], t["W"], t["A"], t["B"], alpha)


def _bwd(t, alpha, rows=None):
    return oracle.lora_group_backward(t["dY"], t["X"], t["W"], t["A"], t["B"], alpha, rows)


def check_single(fwd, bwd):
    t = _group([24], 10, 16, 4, 8.0, 1)
    U, Y = fwd(t, 8.0)
    dU, dX, dA, dB = bwd(t, 8.0)
    U0, Y0 = oracle.lora_forward(t["X"], t["W"][0], t["A"][0], t["B"][0], 8.0)
    g0 = oracle.lora_backward(t["dY"][0], t["X"], t["W"][0], t["A"][0], t["B"][0], 8.0)
    return (np.array_equal(U[0], U0) and np.array_equal(Y[0], Y0) and np.array_equal(dU[0], g0[0])
            and np.array_equal(dX, g0[1]) and np.array_equal(dA[0], g0[2]) and np.array_equal(dB[0], g0[3]))


def check_stacked(fwd, bwd):
    ns, m, k, r, alpha = [16, 24, 8], 9, 32, 3, 6.0
    t = _group(ns, m, k, r, alpha, 2)
    G = len(ns)
    dec = oracle.bf16_bits_to_f64
    Ws = np.concatenate([dec(w) for w in t["W"]])
    As = np.concatenate([dec(a) for a in t["A"]])
    Bbd = np.zeros((sum(ns), G * r))
    dYs = np.concatenate([dec(d) for d in t["dY"]], axis=1)
    off = np.cumsum([0] + ns)
    for g in range(G):
        Bbd[off[g]:off[g + 1], g * r:(g + 1) * r] = dec(t["B"][g])
    s = alpha / r
    Us, Ys = oracle.lora_forward(t["X"], Ws, As, Bbd, s * G * r)
    dUs, dXs, dAs, dBs = oracle.lora_backward(dYs, t["X"], Ws, As, Bbd, s * G * r)
    U, Y = fwd(t, alpha)
    dU, dX, dA, dB = bwd(t, alpha)
    tol = dict(rtol=0, atol=1e-12)
    ok = np.allclose(dXs, dX, **tol)
    for g in range(G):
        ok = ok and np.allclose(Ys[:, off[g]:off[g + 1]], Y[g], **tol)
        ok = ok and np.allclose(Us[:, g * r:(g + 1) * r], U[g], **tol)
        ok = ok and np.allclose(dUs[:, g * r:(g + 1) * r], dU[g], **tol)
        ok = ok and np.allclose(dAs[g * r:(g + 1) * r], dA[g], **tol)
        ok = ok and np.allclose(dBs[off[g]:off[g + 1], g * r:(g + 1) * r], dB[g], **tol)
    return bool(ok)


def check_fd(fwd, bwd):
    alpha = 4.0
    t = _group([6, 4, 8], 5, 8, 2, alpha, 3)
    dec = oracle.bf16_bits_to_f64
    _, dX, dA, dB = bwd(t, alpha)
    base = {"X": dec(t["X"]), "A": [dec(a) for a in t["A"]], "B": [dec(b) for b in t["B"]]}

    def L(tt):
        Y = fwd(tt, alpha)[1]
        return float(sum(np.sum(dec(d) * y) for d, y in zip(t["dY"], Y)))

    h = 2.0 ** -10
    rng = np.random.default_rng(4)
    cases = [("X", None, dX)] + [("A", g, dA[g]) for g in range(3)] + [("B", g, dB[g]) for g in range(3)]
    for name, g, grad in cases:
        for _ in range(4):
            idx = tuple(rng.integers(0, s) for s in grad.shape)
            vals = []
            for sign in (1, -1):
                tt = dict(t)
                if g is None:
                    v = base[name].copy()
                    v[idx] += sign * h
                    tt[name] = v
                else:
                    lst = list(base[name])
                    v = lst[g].copy()
                    v[idx] += sign * h
                    lst[g] = v
                    tt[name] = lst
                vals.append(L(tt))
            fd = (vals[0] - vals[1]) / (2 * h)
            if abs(fd - grad[idx]) > 1e-9 * max(1.0, abs(grad[idx])):
                return False
    return True


def check_brute(fwd, bwd):
    alpha = 3.0
    ns, m, k, r = [2, 4], 3, 4, 2
    t = _group(ns, m, k, r, alpha, 5)
    dec = oracle.bf16_bits_to_f64
    X = dec(t["X"])
    s = alpha / r
    dX = [[0.0] * k for _ in range(m)]
    U, Y, dA, dB = [], [], [], []
    for g, n in enumerate(ns):
        W, A, B, dY = dec(t["W"][g]), dec(t["A"][g]), dec(t["B"][g]), dec(t["dY"][g])
        Ug = [[sum(X[i, l] * A[q, l] for l in range(k)) for q in range(r)] for i in range(m)]
        Y.append([[sum(X[i, l] * W[j, l] for l in range(k)) + s * sum(Ug[i][q] * B[j, q] for q in range(r))
                   for j in range(n)] for i in range(m)])
        dU = [[s * sum(dY[i, j] * B[j, q] for j in range(n)) for q in range(r)] for i in range(m)]
        for i in range(m):
            for l in range(k):
                dX[i][l] += sum(dY[i, j] * W[j, l] for j in range(n)) + sum(dU[i][q] * A[q, l] for q in range(r))
        dA.append([[sum(dU[i][q] * X[i, l] for i in range(m)) for l in range(k)] for q in range(r)])
        dB.append([[s * sum(dY[i, j] * Ug[i][q] for i in range(m)) for q in range(r)] for j in range(n)])
        U.append(Ug)
    Uo, Yo = fwd(t, alpha)
    _, dXo, dAo, dBo = bwd(t, alpha)
    close = lambda a, b: np.allclose(a, np.array(b), rtol=0, atol=1e-12)
    return (close(dXo, dX) and all(close(a, b) for a, b in zip(Uo, U)) and all(close(a, b) for a, b in zip(Yo, Y))
            and all(close(a, b) for a, b in zip(dAo, dA)) and all(close(a, b) for a, b in zip(dBo, dB)))


def check_rows(fwd, bwd):
    t = _group([8, 16], 12, 8, 2, 4.0, 6)
    rows = [0, 5, 11]
    full = bwd(t, 4.0)
    part = bwd(t, 4.0, rows) if bwd is _bwd else None
    return part is None or np.array_equal(part[1], full[1][rows])


CHECKS = [check_single, check_stacked, check_fd, check_brute, check_rows]


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_group_pin(check):
    assert check(_fwd, _bwd)


# ---- planted mistakes (each must fail at least one pin) ---------------------
def _mut_dx_last_only(t, alpha, rows=None):
    dU, dX, dA, dB = _bwd(t, alpha)
    last = oracle.lora_backward(t["dY"][-1], t["X"], t["W"][-1], t["A"][-1], t["B"][-1], alpha)
    return dU, last[1], dA, dB


def _mut_dx_mean(t, alpha, rows=None):
    dU, dX, dA, dB = _bwd(t, alpha)
    return dU, dX / len(t["W"]), dA, dB


def _mut_u_shifted(t, alpha):
    # projection g's rank-r update built from the next projection's U
    U, Y = _fwd(t, alpha)
    dec = oracle.bf16_bits_to_f64
    X = dec(t["X"])
    s = alpha / dec(t["A"][0]).shape[0]
    G = len(U)
    Ym = [X @ dec(t["W"][g]).T + s * U[(g + 1) % G] @ dec(t["B"][g]).T for g in range(G)]
    return U, Ym


def _mut_da_wrong_du(t, alpha, rows=None):
    dU, dX, dA, dB = _bwd(t, alpha)
    X = oracle.bf16_bits_to_f64(t["X"])
    return dU, dX, [dU[0].T @ X for _ in dA], dB


def _mut_dx_without_lora(t, alpha, rows=None):
    dU, dX, dA, dB = _bwd(t, alpha)
    dec = oracle.bf16_bits_to_f64
    return dU, sum(dec(d) @ dec(w) for d, w in zip(t["dY"], t["W"])), dA, dB


MUTANTS = [("dx_last_only", _fwd, _mut_dx_last_only), ("dx_mean", _fwd, _mut_dx_mean),
           ("u_shifted", _mut_u_shifted, _bwd), ("da_wrong_du", _fwd, _mut_da_wrong_du),
           ("dx_without_lora", _fwd, _mut_dx_without_lora)]


@pytest.mark.parametrize("name,fwd,bwd", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_group_mistake(name, fwd, bwd):
    assert not all(check(fwd, bwd) for check in CHECKS)
