"""The fused backward (lora_linear_bwd_fused: dU and the dB partials formed
inside the dX GEMM) against the fp64 oracle, through the C ABI.

Same bars as the other parity tests: relative Frobenius error <= 5e-3 for Y
and dX, <= 1e-2 for dA and dB; bit-exact on integer inputs, where every
partial sum is an exactly representable integer whatever the order.  The
shapes cover the kernel's cases: n a multiple of 64 and k of 256 or not, r a
multiple of 8 or not (two ways of staging B), one to seven 64-wide n stages,
a single dX column tile (every stage then forms dB partials, alternating
between the two sets of four waves), ragged token tails.
"""
import numpy as np
import pytest

import oracle
from lora_synth import CONFIGS, Shape, gen_inputs, gen_ternary_inputs
from gpu_harness import assert_within, compare, run_gpu, sample_rows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2403_11366_amd as lora
    lora.load_library()  # raises if the HIP library is missing: no fallback


def _id(s: Shape):
    return f"{s.name}-m{s.m}n{s.n}k{s.k}r{s.r}"


SHAPES = [
    Shape("fused", 1, 64, 64, 8, 16.0, 1101),
    Shape("fused", 7, 64, 256, 1, 2.0, 1102),
    Shape("fused", 33, 8, 8, 3, 6.0, 1103),
    Shape("fused", 257, 136, 200, 16, 32.0, 1104),
    Shape("fused", 300, 520, 264, 13, 26.0, 1105),
    Shape("fused", 1000, 128, 8, 8, 16.0, 1106),
    Shape("fused", 2051, 4096, 4096, 8, 16.0, 1107),
    Shape("fused", 2000, 4000, 4104, 5, 10.0, 1108),
    Shape("fused", 1500, 3000, 2056, 16, 32.0, 1109),
    Shape("fused", 640, 2048, 1024, 16, 32.0, 1110),
]


@pytest.mark.parametrize("shape", SHAPES, ids=_id)
def test_fused_matches_oracle(shape):
    t = gen_inputs(shape, b_std=0.5)
    out = run_gpu(t, shape, fused=True)
    rows = None if shape.m * shape.n * shape.k < 4e9 else sample_rows(shape.m, shape.seed)
    errs = compare(t, shape, out, rows)
    print(_id(shape), errs)
    assert_within(errs, _id(shape))


@pytest.mark.parametrize("shape", [s for name in ("llama2_7b_q_proj", "llama2_7b_up_proj") for s in CONFIGS[name]],
                         ids=_id)
def test_fused_full_size(shape):
    t = gen_inputs(shape)
    out = run_gpu(t, shape, fused=True)
    errs = compare(t, shape, out, sample_rows(shape.m, shape.seed))
    print(_id(shape), errs)
    assert_within(errs, _id(shape))


EXACT = ([Shape("fexact", 2000, n, 2304, 8, 8.0, 1200 + n) for n in (64, 128, 192, 256, 320, 384, 448)]
         + [Shape("fexact", 2000, n, 2304, r, float(r), 1300 + n) for n, r in ((8, 3), (136, 16), (264, 13))]
         + [Shape("fexact", 257, 1024, 4096, 8, 8.0, 1401), Shape("fexact", 4100, 512, 256, 16, 16.0, 1402),
            Shape("fexact", 2048, 4096, 4096, 8, 8.0, 1403)])


@pytest.mark.parametrize("shape", EXACT, ids=_id)
def test_fused_integer_inputs_bit_exact(shape):
    t = gen_ternary_inputs(shape.m, shape.n, shape.k, shape.r, shape.seed, density=0.1)
    U, Y = oracle.lora_forward(t["X"], t["W"], t["A"], t["B"], shape.alpha)
    dU, dX, dA, dB = oracle.lora_backward(t["dY"], t["X"], t["W"], t["A"], t["B"], shape.alpha)
    assert np.abs(dX).max() <= 256 and np.abs(dU).max() <= 256
    for name, v in (("dU", dU), ("dX", dX), ("dA", dA), ("dB", dB)):
        assert np.array_equal(v, np.round(v)), name
    out = run_gpu(t, shape, fused=True)
    assert np.array_equal(out["dX"], oracle.f64_to_bf16_bits(dX))
    assert np.array_equal(out["dA"].astype(np.float64), dA)
    assert np.array_equal(out["dB"].astype(np.float64), dB)


def test_fused_deterministic_and_close_to_plain():
    shape = Shape("fdet", 1100, 1536, 2048, 16, 32.0, 1501)
    t = gen_inputs(shape, b_std=0.5)
    a = run_gpu(t, shape, fused=True)
    b = run_gpu(t, shape, fused=True)
    for key in ("dX", "dA", "dB"):
        assert np.array_equal(a[key], b[key]), key
    plain = run_gpu(t, shape)
    errs_f = compare(t, shape, a)
    errs_p = compare(t, shape, plain)
    for key in ("dX", "dA", "dB"):   # same accuracy class as the unfused path
        assert errs_f[key] <= 2 * errs_p[key] + 1e-6, (key, errs_f, errs_p)
