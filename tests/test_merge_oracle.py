"""Pins of the oracle's merge (Eq. 1's second form, W0 x + B A x = (W0 + B A) x,
with the LoRA scale s) and of its one-step float64 -> bfloat16 rounding.

  * rne         -- the rounding against its definition: ties go to the even
                   pattern, every result is a nearest bfloat16 value (its two
                   neighbours are not closer), it agrees with the single
                   rounding of float32-exact inputs, and it does not double
                   round (a value just above a tie rounds up).
  * identity    -- the merged weight reproduces the unmerged forward of Eq. 1:
                   X (W + s B A)^T = X W^T + s (X A^T) B^T.
  * unmerge     -- merging then unmerging in float64 returns W.
  * zero        -- B = 0 or A = 0: the stored merge is W bit for bit.
  * hand        -- a hand-worked 2 x 2 example (the one in tests/golden),
                   merged and unmerged.
  * brute       -- scalar loops over the index definition, tiny shapes.
A last test plants plausible mistakes in the merge and checks that a pin
catches each of them.
"""
import numpy as np
import pytest

import oracle
from lora_synth import Shape, gen_inputs


def _bf16_value(bits):
    return oracle.bf16_bits_to_f64(np.asarray(bits, dtype=np.uint16))


def _neighbours(bits):
    """bfloat16 values one pattern below and above (finite, same sign side)."""
    b = np.asarray(bits, dtype=np.int64)
    return _bf16_value((b - 1) & 0xFFFF), _bf16_value((b + 1) & 0xFFFF)


def test_rne_ties_to_even():
    # midpoints between consecutive bfloat16 values in [1, 2): 1 + (2j+1) 2^-8
    j = np.arange(128)
    x = 1.0 + (2 * j + 1) * 2.0 ** -8
    got = oracle.f64_to_bf16_rne(x)
    lower, upper = 0x3F80 + j, 0x3F80 + j + 1     # upper may be 2.0 = 0x4000 when j = 127
    expect = np.where(lower % 2 == 0, lower, upper)
    assert np.array_equal(got.astype(np.int64), expect)
    # the same ties, negative and scaled by powers of two
    for e in (-100, -10, 0, 7, 60):
        xs = -x * 2.0 ** e
        exp_bits = (expect + ((e) << 7)) | 0x8000
        assert np.array_equal(oracle.f64_to_bf16_rne(xs).astype(np.int64), exp_bits)


def test_rne_is_nearest():
    rng = np.random.default_rng(7)
    x = rng.standard_normal(20000) * np.exp2(rng.integers(-60, 60, size=20000))
    bits = oracle.f64_to_bf16_rne(x)
    y = _bf16_value(bits)
    lo, hi = _neighbours(bits)
    d = np.abs(x - y)
    assert np.all(d <= np.abs(x - lo)) and np.all(d <= np.abs(x - hi))
    assert np.all(np.sign(y) == np.sign(x))


def test_rne_matches_single_rounding_of_float32_inputs():
    rng = np.random.default_rng(8)
    x32 = (rng.standard_normal(50000) * 3).astype(np.float32)
    assert np.array_equal(oracle.f64_to_bf16_rne(x32.astype(np.float64)), oracle.f64_to_bf16_bits(x32))


def test_rne_no_double_rounding():
    # 1 + 2^-8 + 2^-30 lies above the tie between 1 and 1 + 2^-7; going through
    # float32 first would land on the tie and round down to 1.
    assert int(oracle.f64_to_bf16_rne(np.array([1.0 + 2.0 ** -8 + 2.0 ** -30]))[0]) == 0x3F81
    assert int(oracle.f64_to_bf16_rne(np.array([1.0 + 2.0 ** -8 - 2.0 ** -30]))[0]) == 0x3F80


def test_rne_subnormal_spacing():
    q = 2.0 ** -133
    x = np.array([3 * q, 3.4 * q, 3.5 * q, 4.5 * q, 127 * q])
    assert oracle.f64_to_bf16_rne(x).tolist() == [3, 3, 4, 4, 127]


def _small(n, k, r, alpha, seed, b_std=0.3):
    return gen_inputs(Shape("pin", 8, n, k, r, alpha, seed), seed=seed, b_std=b_std)


def check_identity(merge_fn):
    for (m, n, k, r, alpha, seed) in [(9, 16, 24, 3, 6.0, 1), (5, 40, 8, 8, 16.0, 2)]:
        t = gen_inputs(Shape("pin", m, n, k, r, alpha, seed), seed=seed, b_std=0.3)
        Wm = merge_fn(t, alpha, 1)
        X = oracle.bf16_bits_to_f64(t["X"])
        _, Y = oracle.lora_forward(t["X"], t["W"], t["A"], t["B"], alpha)
        if np.linalg.norm(X @ Wm.T - Y) > 1e-12 * np.linalg.norm(Y):
            return False
    return True


def check_unmerge(merge_fn):
    t = _small(24, 40, 5, 10.0, 3)
    Wm = merge_fn(t, 10.0, 1)
    t2 = dict(t)
    t2["W"] = Wm
    back = merge_fn(t2, 10.0, -1)
    W = oracle.bf16_bits_to_f64(t["W"])
    return bool(np.max(np.abs(back - W)) <= 1e-14 * np.max(np.abs(W)))


def check_zero(merge_fn):
    t = _small(32, 16, 4, 8.0, 4)
    tb = dict(t)
    tb["B"] = np.zeros_like(t["B"])
    ta = dict(t)
    ta["A"] = np.zeros_like(t["A"])
    W = oracle.bf16_bits_to_f64(t["W"])
    return bool(np.array_equal(merge_fn(tb, 8.0, 1), W) and np.array_equal(merge_fn(ta, 8.0, -1), W))


def check_hand(merge_fn):
    # W = I, A = [[1, 1]], B = [[1], [0]], r = 1, alpha = 2 (s = 2):
    # W + s B A = [[3, 2], [0, 1]];  W - s B A = [[-1, -2], [0, 1]].
    f = oracle.f64_to_bf16_rne
    t = {"W": f(np.eye(2)), "A": f(np.array([[1.0, 1.0]])), "B": f(np.array([[1.0], [0.0]]))}
    return (np.array_equal(merge_fn(t, 2.0, 1), [[3.0, 2.0], [0.0, 1.0]])
            and np.array_equal(merge_fn(t, 2.0, -1), [[-1.0, -2.0], [0.0, 1.0]]))


def check_brute(merge_fn):
    for (n, k, r, alpha, sign, seed) in [(3, 5, 2, 4.0, 1, 5), (4, 2, 3, 1.5, -1, 6)]:
        t = _small(n, k, r, alpha, seed)
        W, A, B = (oracle.bf16_bits_to_f64(t[x]) for x in ("W", "A", "B"))
        s = alpha / r
        ref = np.zeros((n, k))
        for j in range(n):
            for l in range(k):
                acc = 0.0
                for q in range(r):
                    acc += B[j, q] * A[q, l]
                ref[j, l] = W[j, l] + sign * s * acc
        if np.max(np.abs(merge_fn(t, alpha, sign) - ref)) > 1e-12:
            return False
    return True


CHECKS = [check_identity, check_unmerge, check_zero, check_hand, check_brute]


def _oracle_merge(t, alpha, sign):
    return oracle.lora_merged_weight(t["W"], t["A"], t["B"], alpha, sign)


@pytest.mark.parametrize("check", CHECKS, ids=lambda c: c.__name__)
def test_merge_pin(check):
    assert check(_oracle_merge)


def test_stored_merge_rounds_the_float64_merge():
    t = _small(64, 48, 8, 16.0, 9)
    bits = oracle.lora_merge_bf16(t["W"], t["A"], t["B"], 16.0, 1)
    assert np.array_equal(bits, oracle.f64_to_bf16_rne(_oracle_merge(t, 16.0, 1)))


def _d(t):
    return {x: oracle.bf16_bits_to_f64(t[x]) if np.asarray(t[x]).dtype == np.uint16 else np.asarray(t[x])
            for x in ("W", "A", "B")}


def _mut_no_scale(t, alpha, sign):
    d = _d(t)
    return d["W"] + sign * (d["B"] @ d["A"])


def _mut_sign_ignored(t, alpha, sign):
    d = _d(t)
    return d["W"] + (alpha / d["A"].shape[0]) * (d["B"] @ d["A"])


def _mut_scale_inverted(t, alpha, sign):
    d = _d(t)
    return d["W"] + sign * (d["A"].shape[0] / alpha) * (d["B"] @ d["A"])


def _mut_rank_shift(t, alpha, sign):
    d = _d(t)
    return d["W"] + sign * (alpha / d["A"].shape[0]) * (d["B"] @ np.roll(d["A"], 1, axis=0))


def _mut_scale_squared(t, alpha, sign):
    d = _d(t)
    s = alpha / d["A"].shape[0]
    return d["W"] + sign * s * s * (d["B"] @ d["A"])


MUTANTS = [_mut_no_scale, _mut_sign_ignored, _mut_scale_inverted, _mut_rank_shift, _mut_scale_squared]


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda f: f.__name__)
def test_pins_catch_planted_merge_mistake(mutant):
    assert not all(check(mutant) for check in CHECKS)
