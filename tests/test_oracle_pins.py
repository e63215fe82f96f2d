"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Every check takes the forward/backward callables as arguments, so the last
test can plant plausible mistakes in the oracle (on the CPU) and confirm that
at least one pin fails for each of them.

Pins:
  * golden    -- two hand-worked examples (tests/golden/hand_examples.txt),
                 computed by hand from Eq. 1 and its merged form.
  * merge     -- Eq. 1's second line: Y = X (W + s B A)^T, and the merged
                 backward dX = dY (W + s B A).
  * eq1_s1    -- with alpha = r (the paper's defaults LORA_R = LORA_ALPHA = 16,
                 Listing 3) the scale is 1 and Y is Eq. 1 exactly as printed.
  * b_zero    -- the paper's initialisation B = 0 (Section 3): Y = X W^T
                 exactly, dU = 0 and dA = 0 exactly.
  * a_zero    -- A = 0: U = 0, dB = 0 exactly, Y = X W^T.
  * fd        -- central finite differences of L = <dY, Y> in every entry of
                 X, A and B.  L is affine in each single entry, so the
                 difference quotient is exact up to fp64 rounding.
  * brute     -- scalar Python loops over the index definitions, tiny shapes.
  * closed    -- dA = s B^T dY^T X and dB = s dY^T X A^T, associated differently.
"""
import os

import numpy as np
import pytest

import oracle
from lora_synth import Shape, gen_inputs

HERE = os.path.dirname(os.path.abspath(__file__))


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    if nb == 0.0:
        return 0.0 if np.linalg.norm(a) == 0.0 else np.inf
    return float(np.linalg.norm(a - b) / nb)


def load_golden():
    path = os.path.join(HERE, "golden", "hand_examples.txt")
    examples, cur, lines = [], None, []
    with open(path) as f:
        for raw in f:
            s = raw.split("#", 1)[0].strip()
            if s:
                lines.append(s)
    i = 0
    while i < len(lines):
        tok = lines[i].split()
        if tok[0] == "example":
            cur = {"name": tok[1], "m": int(tok[2]), "n": int(tok[3]), "k": int(tok[4]),
                   "r": int(tok[5]), "alpha": float(tok[6]), "t": {}}
            examples.append(cur)
            i += 1
            continue
        name, rows, cols = tok[0], int(tok[1]), int(tok[2])
        vals = [list(map(float, lines[i + 1 + j].split())) for j in range(rows)]
        arr = np.array(vals, dtype=np.float64).reshape(rows, cols)
        cur["t"][name] = arr
        i += 1 + rows
    return examples


# ----------------------------------------------------------------------------
# checks, parameterised by the implementation under test

def check_golden(fwd, bwd):
    for ex in load_golden():
        t = ex["t"]
        U, Y = fwd(t["X"], t["W"], t["A"], t["B"], ex["alpha"])
        dU, dX, dA, dB = bwd(t["dY"], t["X"], t["W"], t["A"], t["B"], ex["alpha"])
        for name, got in (("U", U), ("Y", Y), ("dU", dU), ("dX", dX), ("dA", dA), ("dB", dB)):
            assert np.array_equal(np.asarray(got), t[name]), (ex["name"], name, got, t[name])


def _small_inputs(m, n, k, r, alpha, seed, b_std=0.3):
    d = gen_inputs(Shape("pin", m, n, k, r, alpha, seed), b_std=b_std)
    return {key: oracle.bf16_bits_to_f64(v) for key, v in d.items()}


def check_merge(fwd, bwd):
    for (m, n, k, r, alpha, seed) in [(7, 12, 9, 3, 6.0, 1), (16, 8, 24, 4, 16.0, 2),
                                      (5, 6, 6, 2, 1.0, 3)]:
        t = _small_inputs(m, n, k, r, alpha, seed)
        s = alpha / r
        Wm = t["W"] + s * (t["B"] @ t["A"])        # merged weight, Eq. 1 second line
        U, Y = fwd(t["X"], t["W"], t["A"], t["B"], alpha)
        assert rel(Y, t["X"] @ Wm.T) <= 1e-12
        dU, dX, dA, dB = bwd(t["dY"], t["X"], t["W"], t["A"], t["B"], alpha)
        assert rel(dX, t["dY"] @ Wm) <= 1e-12


def check_eq1_s1(fwd, bwd):
    t = _small_inputs(6, 5, 7, 16, 16.0, 4)       # alpha = r = 16: scale 1
    U, Y = fwd(t["X"], t["W"], t["A"], t["B"], 16.0)
    # W0 x + B A x, row by row, as printed in Eq. 1 (b0 = 0)
    printed = np.stack([t["W"] @ x + t["B"] @ (t["A"] @ x) for x in t["X"]])
    assert rel(Y, printed) <= 1e-12


def check_b_zero(fwd, bwd):
    t = _small_inputs(9, 10, 12, 4, 8.0, 5)
    Bz = np.zeros_like(t["B"])
    U, Y = fwd(t["X"], t["W"], t["A"], Bz, 8.0)
    assert np.array_equal(Y, t["X"] @ t["W"].T)
    dU, dX, dA, dB = bwd(t["dY"], t["X"], t["W"], t["A"], Bz, 8.0)
    assert not np.any(dU) and not np.any(dA)
    assert np.array_equal(dX, t["dY"] @ t["W"])
    assert rel(U, t["X"] @ t["A"].T) <= 1e-15


def check_a_zero(fwd, bwd):
    t = _small_inputs(9, 10, 12, 4, 8.0, 6)
    Az = np.zeros_like(t["A"])
    U, Y = fwd(t["X"], t["W"], Az, t["B"], 8.0)
    assert not np.any(U)
    assert np.array_equal(Y, t["X"] @ t["W"].T)
    dU, dX, dA, dB = bwd(t["dY"], t["X"], t["W"], Az, t["B"], 8.0)
    assert not np.any(dB)


def check_fd(fwd, bwd):
    h = 2.0 ** -10
    for (m, n, k, r, alpha, seed) in [(3, 4, 5, 2, 4.0, 7), (2, 3, 4, 3, 3.0, 8)]:
        t = _small_inputs(m, n, k, r, alpha, seed)
        dU, dX, dA, dB = bwd(t["dY"], t["X"], t["W"], t["A"], t["B"], alpha)

        def L(X, A, B):
            return float(np.sum(t["dY"] * fwd(X, t["W"], A, B, alpha)[1]))

        for name, grad in (("X", dX), ("A", dA), ("B", dB)):
            base = t[name]
            for idx in np.ndindex(*base.shape):
                args = {"X": t["X"], "A": t["A"], "B": t["B"]}
                p, q = base.copy(), base.copy()
                p[idx] += h
                q[idx] -= h
                args[name] = p
                lp = L(args["X"], args["A"], args["B"])
                args[name] = q
                lq = L(args["X"], args["A"], args["B"])
                fd = (lp - lq) / (2 * h)
                assert abs(fd - grad[idx]) <= 1e-9 * max(1.0, abs(fd)), (name, idx, fd, grad[idx])


def check_brute(fwd, bwd):
    m, n, k, r, alpha = 3, 4, 5, 2, 6.0
    t = _small_inputs(m, n, k, r, alpha, 9)
    X, W, A, B, dY = (t[x].tolist() for x in ("X", "W", "A", "B", "dY"))
    s = alpha / r
    U = [[sum(X[i][l] * A[q][l] for l in range(k)) for q in range(r)] for i in range(m)]
    Y = [[sum(X[i][l] * W[j][l] for l in range(k)) + s * sum(U[i][q] * B[j][q] for q in range(r))
          for j in range(n)] for i in range(m)]
    dU = [[s * sum(dY[i][j] * B[j][q] for j in range(n)) for q in range(r)] for i in range(m)]
    dX = [[sum(dY[i][j] * W[j][l] for j in range(n)) + sum(dU[i][q] * A[q][l] for q in range(r))
           for l in range(k)] for i in range(m)]
    dB = [[s * sum(dY[i][j] * U[i][q] for i in range(m)) for q in range(r)] for j in range(n)]
    dA = [[sum(dU[i][q] * X[i][l] for i in range(m)) for l in range(k)] for q in range(r)]
    gU, gY = fwd(t["X"], t["W"], t["A"], t["B"], alpha)
    gdU, gdX, gdA, gdB = bwd(t["dY"], t["X"], t["W"], t["A"], t["B"], alpha)
    for ref, got in ((U, gU), (Y, gY), (dU, gdU), (dX, gdX), (dA, gdA), (dB, gdB)):
        assert rel(got, ref) <= 1e-13


def check_closed(fwd, bwd):
    m, n, k, r, alpha = 11, 7, 13, 5, 10.0
    t = _small_inputs(m, n, k, r, alpha, 10)
    s = alpha / r
    dU, dX, dA, dB = bwd(t["dY"], t["X"], t["W"], t["A"], t["B"], alpha)
    assert rel(dA, s * (t["B"].T @ (t["dY"].T @ t["X"]))) <= 1e-12
    assert rel(dB, s * ((t["dY"].T @ t["X"]) @ t["A"].T)) <= 1e-12


ALL_CHECKS = [check_golden, check_merge, check_eq1_s1, check_b_zero, check_a_zero,
              check_fd, check_brute, check_closed]


# ----------------------------------------------------------------------------
# the oracle against every pin

def _oracle_fwd(X, W, A, B, alpha):
    return oracle.lora_forward(X, W, A, B, alpha)


def _oracle_bwd(dY, X, W, A, B, alpha):
    return oracle.lora_backward(dY, X, W, A, B, alpha)


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_oracle_pin(check):
    check(_oracle_fwd, _oracle_bwd)


def test_bf16_decode_exact():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x8000, 0x4049, 0x7F7F, 0x0001], dtype=np.uint16)
    vals = oracle.bf16_bits_to_f64(bits)
    assert vals[0] == 1.0 and vals[1] == -1.0 and vals[2] == 0.0
    assert np.signbit(vals[3]) and vals[3] == 0.0
    assert vals[4] == 3.140625
    assert vals[5] == (2 - 2 ** -7) * 2.0 ** 127
    assert vals[6] == 2.0 ** -133


def test_rows_variants_match_full():
    t = gen_inputs(Shape("rows", 37, 24, 40, 8, 16.0, 11))
    rows = [0, 5, 17, 36]
    U, Y = oracle.lora_forward(t["X"], t["W"], t["A"], t["B"], 16.0)
    Ur, Yr = oracle.lora_forward_rows(t["X"], t["W"], t["A"], t["B"], 16.0, rows)
    assert np.array_equal(Ur, U[rows]) and np.array_equal(Yr, Y[rows])
    dU, dX, dA, dB = oracle.lora_backward(t["dY"], t["X"], t["W"], t["A"], t["B"], 16.0)
    dUr, dXr, dAr, dBr = oracle.lora_backward_rows(t["dY"], t["X"], t["W"], t["A"], t["B"], 16.0, rows)
    assert np.array_equal(dUr, dU) and np.array_equal(dAr, dA) and np.array_equal(dBr, dB)
    assert rel(dXr, dX[rows]) <= 1e-15


# ----------------------------------------------------------------------------
# planted mistakes: each must trip at least one pin

def _mut_fwd_no_scale(X, W, A, B, alpha):
    U, _ = oracle.lora_forward(X, W, A, B, alpha)
    return U, np.asarray(X) @ np.asarray(W).T + U @ np.asarray(B).T


def _mut_fwd_scale_inverted(X, W, A, B, alpha):
    r = np.asarray(A).shape[0]
    U, _ = oracle.lora_forward(X, W, A, B, alpha)
    return U, np.asarray(X) @ np.asarray(W).T + (r / alpha) * (U @ np.asarray(B).T)


def _mut_fwd_w_not_transposed(X, W, A, B, alpha):
    U, Y = oracle.lora_forward(X, W, A, B, alpha)
    X, W = np.asarray(X), np.asarray(W)
    if X.shape[1] == W.shape[0] == W.shape[1]:
        Y = Y - X @ W.T + X @ W
    return U, Y


def _mut_fwd_lora_sign(X, W, A, B, alpha):
    U, Y = oracle.lora_forward(X, W, A, B, alpha)
    base = np.asarray(X) @ np.asarray(W).T
    return U, base - (Y - base)


def _bwd_parts(dY, X, W, A, B, alpha):
    return oracle.lora_backward(dY, X, W, A, B, alpha)


def _mut_bwd_dx_no_lora(dY, X, W, A, B, alpha):
    dU, dX, dA, dB = _bwd_parts(dY, X, W, A, B, alpha)
    return dU, np.asarray(dY) @ np.asarray(W), dA, dB


def _mut_bwd_db_no_scale(dY, X, W, A, B, alpha):
    dU, dX, dA, dB = _bwd_parts(dY, X, W, A, B, alpha)
    return dU, dX, dA, dB / (alpha / np.asarray(A).shape[0])


def _mut_bwd_da_double_scale(dY, X, W, A, B, alpha):
    dU, dX, dA, dB = _bwd_parts(dY, X, W, A, B, alpha)
    return dU, dX, dA * (alpha / np.asarray(A).shape[0]), dB


def _mut_bwd_du_no_scale(dY, X, W, A, B, alpha):
    dU, dX, dA, dB = _bwd_parts(dY, X, W, A, B, alpha)
    s = alpha / np.asarray(A).shape[0]
    dU2 = dU / s
    return dU2, np.asarray(dY) @ np.asarray(W) + dU2 @ np.asarray(A), dU2.T @ np.asarray(X), dB


def _mut_bwd_dx_lora_sign(dY, X, W, A, B, alpha):
    dU, dX, dA, dB = _bwd_parts(dY, X, W, A, B, alpha)
    base = np.asarray(dY) @ np.asarray(W)
    return dU, base - (dX - base), dA, dB


def _mut_bwd_da_uses_x_row_shift(dY, X, W, A, B, alpha):
    dU, dX, dA, dB = _bwd_parts(dY, X, W, A, B, alpha)
    Xs = np.roll(np.asarray(X, dtype=np.float64), 1, axis=0)
    return dU, dX, dU.T @ Xs, dB


def _mut_bwd_db_transposed_reduction(dY, X, W, A, B, alpha):
    dU, dX, dA, dB = _bwd_parts(dY, X, W, A, B, alpha)
    s = alpha / np.asarray(A).shape[0]
    U = np.asarray(X, dtype=np.float64) @ np.asarray(A, dtype=np.float64).T
    dYr = np.asarray(dY, dtype=np.float64)[::-1]
    return dU, dX, dA, s * (dYr.T @ U)


MUTANTS = [
    ("fwd_no_scale", _mut_fwd_no_scale, _oracle_bwd),
    ("fwd_scale_inverted", _mut_fwd_scale_inverted, _oracle_bwd),
    ("fwd_w_not_transposed", _mut_fwd_w_not_transposed, _oracle_bwd),
    ("fwd_lora_sign", _mut_fwd_lora_sign, _oracle_bwd),
    ("bwd_dx_no_lora", _oracle_fwd, _mut_bwd_dx_no_lora),
    ("bwd_db_no_scale", _oracle_fwd, _mut_bwd_db_no_scale),
    ("bwd_da_double_scale", _oracle_fwd, _mut_bwd_da_double_scale),
    ("bwd_du_no_scale", _oracle_fwd, _mut_bwd_du_no_scale),
    ("bwd_dx_lora_sign", _oracle_fwd, _mut_bwd_dx_lora_sign),
    ("bwd_da_row_shift", _oracle_fwd, _mut_bwd_da_uses_x_row_shift),
    ("bwd_db_wrong_pairing", _oracle_fwd, _mut_bwd_db_transposed_reduction),
]


@pytest.mark.parametrize("name,fwd,bwd", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(name, fwd, bwd):
    failed = []
    for check in ALL_CHECKS:
        try:
            check(fwd, bwd)
        except AssertionError:
            failed.append(check.__name__)
    assert failed, f"planted mistake {name} passed every pin"


def test_f64_to_bf16_bits_rounding():
    """The oracle's bf16 encoder used by the bit-exact GPU tests: exact for
    small integers, ties to even (1 + 2^-8 -> 1, 1 + 3*2^-8 -> 1 + 2^-6)."""
    vals = np.array([0.0, 1.0, -3.0, 256.0, 255.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8], dtype=np.float64)
    got = oracle.bf16_bits_to_f64(oracle.f64_to_bf16_bits(vals))
    assert got.tolist() == [0.0, 1.0, -3.0, 256.0, 255.0, 1.0, 1 + 2 ** -6]


# ----------------------------------------------------------------------------
# the rank-r activation U = X A^T on its own (oracle.lora_rank_activation, the
# U reference of the GPU tests), pinned by checks parameterised by the function

def check_u_golden(u_fn):
    """The hand-worked U of tests/golden (computed by hand from Eq. 1's A x term)."""
    for ex in load_golden():
        t = ex["t"]
        assert np.array_equal(np.asarray(u_fn(t["X"], t["A"])), t["U"]), ex["name"]


def check_u_brute(u_fn):
    """Scalar loops over the index definition U[i][t] = sum_l X[i][l] A[t][l]."""
    t = _small_inputs(4, 3, 6, 3, 6.0, 12)
    X, A = t["X"].tolist(), t["A"].tolist()
    ref = [[sum(X[i][l] * A[q][l] for l in range(6)) for q in range(3)] for i in range(4)]
    assert rel(u_fn(t["X"], t["A"]), ref) <= 1e-14


def check_u_through_forward(u_fn):
    """Another route: with W = 0 and B the identity (n = r), Eq. 1 gives
    Y = s U, so U = Y / s from the (separately pinned) forward."""
    m, k, r, alpha = 9, 11, 4, 12.0
    t = _small_inputs(m, r, k, r, alpha, 13)
    _, Y = oracle.lora_forward(t["X"], np.zeros((r, k)), t["A"], np.eye(r), alpha)
    assert rel(u_fn(t["X"], t["A"]), Y / (alpha / r)) <= 1e-14


def check_u_linear_in_x(u_fn):
    """U is linear in each row of X: the change of U[i] for a unit change of
    X[i][l] is column l of A, and other rows do not move."""
    t = _small_inputs(5, 3, 7, 3, 6.0, 14)
    base = np.asarray(u_fn(t["X"], t["A"]), dtype=np.float64)
    for i, l in ((0, 0), (2, 5), (4, 6)):
        X2 = t["X"].copy()
        X2[i, l] += 1.0
        d = np.asarray(u_fn(X2, t["A"]), dtype=np.float64) - base
        expect = np.zeros_like(base)
        expect[i] = t["A"][:, l]
        assert np.allclose(d, expect, rtol=0, atol=1e-12), (i, l)


U_CHECKS = [check_u_golden, check_u_brute, check_u_through_forward, check_u_linear_in_x]


@pytest.mark.parametrize("check", U_CHECKS, ids=lambda c: c.__name__)
def test_rank_activation_pin(check):
    check(oracle.lora_rank_activation)


def test_rank_activation_is_the_forward_u():
    t = gen_inputs(Shape("u", 70, 48, 136, 13, 26.0, 15))
    assert np.array_equal(oracle.lora_rank_activation(t["X"], t["A"]),
                          oracle.lora_forward(t["X"], t["W"], t["A"], t["B"], 26.0)[0])


U_MUTANTS = [
    ("u_a_rows_rolled", lambda X, A: oracle.lora_rank_activation(X, np.roll(np.asarray(A), 1, axis=0))),
    ("u_x_rows_reversed", lambda X, A: oracle.lora_rank_activation(np.asarray(X)[::-1], A)),
    ("u_a_columns_reversed", lambda X, A: oracle.lora_rank_activation(X, np.asarray(A)[:, ::-1])),
    ("u_scaled", lambda X, A: 2.0 * oracle.lora_rank_activation(X, A)),
    ("u_sign", lambda X, A: -oracle.lora_rank_activation(X, A)),
]


@pytest.mark.parametrize("name,fn", U_MUTANTS, ids=[m[0] for m in U_MUTANTS])
def test_rank_activation_pins_catch_planted_mistake(name, fn):
    failed = []
    for check in U_CHECKS:
        try:
            check(fn)
        except AssertionError:
            failed.append(check.__name__)
    assert failed, f"planted mistake {name} passed every U pin"
