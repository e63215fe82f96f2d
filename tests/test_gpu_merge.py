"""GPU parity of lora_linear_merge (through the C ABI) against the fp64 oracle.

The kernel accumulates the rank-r product in fp32, forms W + sign s B A in
fp32 and rounds once to bf16; the oracle rounds the exact float64 value once.
So every element must lie within the error bound of that arithmetic: half a
bf16 spacing at the result plus the fp32 accumulation bound
(r + 2) 2^-24 (|W| + s |B| |A|).  The two roundings can disagree only where
the exact value is that close to a bf16 rounding boundary, so at most 1e-3 of
the elements may differ from the oracle's bits, and the relative Frobenius
error must be within the tolerance of Y (5e-3).  Integer inputs whose merge is
exactly representable must match bit for bit.
"""
import numpy as np
import pytest

import oracle
from lora_synth import Shape, gen_inputs
from gpu_harness import TOL_Y, rel

pytestmark = pytest.mark.gpu


def run_merge(t, alpha, sign, in_place=False, poison=True):
    import torch
    import paper_2403_11366_amd as lora
    from paper_2403_11366_amd.device_io import bits_to_device, device_to_bits
    W, A, B = (bits_to_device(t[x]) for x in ("W", "A", "B"))
    if in_place:
        out = W
    else:
        out = torch.empty_like(W)
        if poison:
            out.fill_(float("nan"))
    lora.lora_linear_merge(W, A, B, out, alpha, sign)
    torch.cuda.synchronize()
    return device_to_bits(out)


def half_spacing(x):
    """Half the distance between consecutive bf16 values around x (normal range;
    2^-134 below it)."""
    _, e = np.frexp(np.asarray(x, dtype=np.float64))
    return np.ldexp(1.0, np.maximum(e, -125) - 9)


def check(t, alpha, sign, got):
    ref_bits = oracle.lora_merge_bf16(t["W"], t["A"], t["B"], alpha, sign)
    ref = oracle.lora_merged_weight(t["W"], t["A"], t["B"], alpha, sign)
    W, A, B = (oracle.bf16_bits_to_f64(t[x]) for x in ("W", "A", "B"))
    r = A.shape[0]
    s = alpha / r
    g = oracle.bf16_bits_to_f64(got)
    bound = half_spacing(g) + (r + 2) * 2.0 ** -24 * (np.abs(W) + s * (np.abs(B) @ np.abs(A)))
    excess = float(np.max(np.abs(g - ref) / bound))
    frac = float(np.mean(got != ref_bits))
    e = rel(g, ref)
    print(f"error / bound <= {excess:.3f}, differing bits {frac:.2e}, rel {e:.2e}", flush=True)
    assert excess <= 1.0
    assert frac <= 1e-3
    assert e <= TOL_Y


SHAPES = [  # (n, k, r, alpha): tiles of 128 x 128, ragged edges, every padded rank
    (8, 8, 1, 2.0), (64, 64, 8, 16.0), (200, 136, 5, 10.0), (256, 384, 16, 32.0),
    (520, 264, 33, 66.0), (1024, 1024, 64, 128.0), (136, 1000, 48, 96.0),
]


@pytest.mark.parametrize("n,k,r,alpha", SHAPES)
@pytest.mark.parametrize("sign", [1, -1])
def test_merge_parity(n, k, r, alpha, sign):
    print(f"merge n={n} k={k} r={r} sign={sign}", flush=True)
    t = gen_inputs(Shape("merge", 8, n, k, r, alpha, 11), seed=11 + r, b_std=0.3)
    check(t, alpha, sign, run_merge(t, alpha, sign))


@pytest.mark.parametrize("name,n,k,r,alpha", [("llama2_7b_q_proj", 4096, 4096, 8, 16.0),
                                              ("llama2_7b_down_proj", 4096, 11008, 64, 128.0),
                                              ("llama2_13b_gate_proj", 13824, 5120, 8, 16.0)])
def test_merge_full_size(name, n, k, r, alpha):
    print(f"merge {name}", flush=True)
    t = gen_inputs(Shape(name, 8, n, k, r, alpha, 12), seed=12, b_std=0.02)
    check(t, alpha, 1, run_merge(t, alpha, 1))


def test_merge_in_place_matches_out_of_place():
    t = gen_inputs(Shape("merge", 8, 384, 520, 24, 48.0, 13), seed=13, b_std=0.3)
    a = run_merge(t, 48.0, 1)
    b = run_merge(t, 48.0, 1, in_place=True)
    assert np.array_equal(a, b)


def test_merge_zero_adapter_is_identity():
    t = gen_inputs(Shape("merge", 8, 264, 392, 12, 24.0, 14), seed=14)
    t["B"] = np.zeros_like(t["B"])
    assert np.array_equal(run_merge(t, 24.0, 1), t["W"])
    assert np.array_equal(run_merge(t, 24.0, -1), t["W"])


def test_merge_integer_exact():
    # small integers: every product and sum is exact in fp32, |W'| < 256 is exact in bf16
    rng = np.random.default_rng(15)
    n, k, r = 392, 264, 7
    f = oracle.f64_to_bf16_rne
    t = {"W": f(rng.integers(-20, 21, size=(n, k)).astype(np.float64)),
         "A": f(rng.integers(-2, 3, size=(r, k)).astype(np.float64)),
         "B": f(rng.integers(-2, 3, size=(n, r)).astype(np.float64))}
    for sign in (1, -1):
        got = run_merge(t, 2.0 * r, sign)   # s = 2
        assert np.array_equal(got, oracle.lora_merge_bf16(t["W"], t["A"], t["B"], 2.0 * r, sign))


def test_merge_deterministic():
    t = gen_inputs(Shape("merge", 8, 512, 512, 16, 32.0, 16), seed=16, b_std=0.3)
    assert np.array_equal(run_merge(t, 32.0, 1), run_merge(t, 32.0, 1))
