"""Seeded random shapes through the C ABI against the fp64 oracle: token
counts, widths and depths drawn anywhere in their ranges (ragged tails at
every position, the plans' tile and split choices at their boundaries) and
ranks 1 .. 64, for the plain, dropout and grouped entry points.  The shapes
are drawn once from a fixed seed, so every run checks the same cases.
"""
import numpy as np
import pytest

from lora_synth import Shape, gen_inputs, gen_keep_mask
from gpu_harness import assert_within, compare, run_gpu
from test_gpu_dropout import check as check_dropout, run_dropout
from test_gpu_group import _group, check as check_group, run_group

pytestmark = pytest.mark.gpu


def _draw(n_cases, seed, k_multiple=8):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n_cases):
        m = int(rng.integers(1, 3001))
        n = 8 * int(rng.integers(1, 385))                  # 8 .. 3072
        k = k_multiple * int(rng.integers(1, 3072 // k_multiple + 1))
        r = int(rng.integers(1, 65))
        out.append(Shape("rand", m, n, k, r, 2.0 * r, 700 + 10 * seed + i))
    return out


PLAIN = _draw(40, 1)
DROP = _draw(16, 2, k_multiple=64)


def _id(s):
    return f"m{s.m}n{s.n}k{s.k}r{s.r}"


@pytest.mark.parametrize("shape", PLAIN, ids=_id)
def test_random_plain(shape):
    print(_id(shape), flush=True)
    t = gen_inputs(shape, b_std=0.5)
    assert_within(compare(t, shape, run_gpu(t, shape)), _id(shape))


@pytest.mark.parametrize("shape", DROP, ids=_id)
def test_random_dropout(shape):
    print(_id(shape), flush=True)
    p = 0.1
    t = gen_inputs(shape, b_std=0.5)
    keep = gen_keep_mask(shape.m, shape.k, p, shape.seed + 3)
    check_dropout(t, shape, keep, p, run_dropout(t, shape, keep, p))


def _groups(n_cases, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n_cases):
        g = int(rng.integers(2, 5))
        ns = [8 * int(rng.integers(1, 257)) for _ in range(g)]   # 8 .. 2048 each
        m = int(rng.integers(1, 2501))
        k = 8 * int(rng.integers(1, 257))
        r = int(rng.integers(1, 65))
        out.append((ns, m, k, r))
    return out


GROUPS = _groups(16, 3)


@pytest.mark.parametrize("ns,m,k,r", GROUPS, ids=[f"G{len(c[0])}-m{c[1]}k{c[2]}r{c[3]}" for c in GROUPS])
def test_random_group(ns, m, k, r):
    print(f"group ns={ns} m={m} k={k} r={r}", flush=True)
    alpha = 2.0 * r
    t = _group(ns, m, k, r, alpha, 900 + m % 97)
    check_group(t, alpha, run_group(t, m, k, r, alpha))
