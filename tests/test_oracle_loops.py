"""The oracle's plain-loop form (oracle/lora_loops.c, float64 loops over the
index definitions) against every pin of the oracle (tests/test_oracle_pins.py:
the hand-worked examples, the merge identity, Eq. 1 at s = 1, the B = 0 and
A = 0 invariants, finite differences, scalar Python loops, closed forms), and
against the numpy form on seeded bf16 inputs (the two evaluate the same
definition in different association orders, so they agree to float64
rounding)."""
import numpy as np
import pytest

import oracle
from oracle import loops
from lora_synth import Shape, gen_inputs
from test_oracle_pins import ALL_CHECKS, MUTANTS, rel


def _fwd(X, W, A, B, alpha):
    return loops.lora_forward_loops(X, W, A, B, alpha, threads=2)


def _bwd(dY, X, W, A, B, alpha):
    return loops.lora_backward_loops(dY, X, W, A, B, alpha, threads=2)


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_loops_pass_every_pin(check):
    check(_fwd, _bwd)


@pytest.mark.parametrize("shape", [Shape("lp", 37, 24, 40, 8, 16.0, 21), Shape("lp", 130, 264, 200, 13, 26.0, 22),
                                   Shape("lp", 64, 512, 512, 64, 128.0, 23)], ids=lambda s: f"m{s.m}n{s.n}k{s.k}r{s.r}")
def test_loops_match_numpy_form(shape):
    t = gen_inputs(shape)
    U, Y = oracle.lora_forward(t["X"], t["W"], t["A"], t["B"], shape.alpha)
    Ul, Yl = loops.lora_forward_loops(t["X"], t["W"], t["A"], t["B"], shape.alpha, threads=4)
    ref = oracle.lora_backward(t["dY"], t["X"], t["W"], t["A"], t["B"], shape.alpha)
    got = loops.lora_backward_loops(t["dY"], t["X"], t["W"], t["A"], t["B"], shape.alpha, threads=4)
    assert rel(Ul, U) <= 1e-13 and rel(Yl, Y) <= 1e-13
    for g, r_ in zip(got, ref):
        assert rel(g, r_) <= 1e-13


def test_loops_thread_count_does_not_change_results():
    t = gen_inputs(Shape("lp", 50, 40, 72, 5, 10.0, 24))
    a = loops.lora_backward_loops(t["dY"], t["X"], t["W"], t["A"], t["B"], 10.0, threads=1)
    b = loops.lora_backward_loops(t["dY"], t["X"], t["W"], t["A"], t["B"], 10.0, threads=3)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
