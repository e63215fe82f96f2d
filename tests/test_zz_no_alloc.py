"""lora_linear_bwd_noalloc (the backward whose workspace is the library's own
per-GPU scratch array) against lora_linear_bwd with a caller workspace,
through the C ABI: two calls in a row, the second on a smaller problem, each
bit-identical to the workspace entry point (same kernels, fixed-order sums),
and the first also within the oracle's tolerances."""
import numpy as np
import pytest

from lora_synth import Shape, gen_inputs
from gpu_harness import assert_within, compare, sample_rows

pytestmark = pytest.mark.gpu


def _run(shape, noalloc: bool):
    import torch
    import paper_2403_11366_amd as lora
    from paper_2403_11366_amd.device_io import bits_to_device, device_to_bits
    m, n, k, r = shape.m, shape.n, shape.k, shape.r
    t = gen_inputs(shape, b_std=0.3)
    d = {key: bits_to_device(v) for key, v in t.items()}
    Y = torch.empty((m, n), dtype=torch.bfloat16, device="cuda")
    U = torch.empty((m, r), dtype=torch.float32, device="cuda")
    dX = torch.full((m, k), float("nan"), dtype=torch.bfloat16, device="cuda")
    dA = torch.full((r, k), float("nan"), dtype=torch.float32, device="cuda")
    dB = torch.full((n, r), float("nan"), dtype=torch.float32, device="cuda")
    lora.lora_linear_fwd(d["X"], d["W"], d["A"], d["B"], Y, U, shape.alpha)
    if noalloc:
        lora.lora_linear_bwd_noalloc(d["dY"], d["X"], d["W"], d["A"], d["B"], U, dX, dA, dB, shape.alpha)
    else:
        ws = torch.full((lora.lora_linear_bwd_workspace_size(m, n, k, r),), 0xFF, dtype=torch.uint8, device="cuda")
        lora.lora_linear_bwd(d["dY"], d["X"], d["W"], d["A"], d["B"], U, dX, dA, dB, ws, shape.alpha)
    torch.cuda.synchronize()
    return t, {"Y": device_to_bits(Y), "U": U.cpu().numpy(), "dX": device_to_bits(dX),
               "dA": dA.cpu().numpy(), "dB": dB.cpu().numpy()}


def test_noalloc_matches_workspace_entry_point_twice():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    # the larger call first (7B down_proj: the largest workspace, 20.75 MiB),
    # then a smaller ragged one that reuses the same scratch
    for shape in (Shape("noalloc_big", 8192, 4096, 11008, 64, 128.0, 3000),
                  Shape("noalloc_small", 1000, 1032, 520, 13, 26.0, 3001)):
        print(f"noalloc {shape}", flush=True)
        t, got = _run(shape, noalloc=True)
        _, ref = _run(shape, noalloc=False)
        for key in ("dX", "dA", "dB"):
            assert np.array_equal(got[key].view(np.uint8), ref[key].view(np.uint8)), (shape.name, key)
        rows = sample_rows(shape.m, shape.seed) if shape.m * shape.n * shape.k > 4e9 else None
        assert_within(compare(t, shape, got, rows), shape.name)


def test_noalloc_refuses_shapes_beyond_its_scratch():
    import torch
    import paper_2403_11366_amd as lora
    from paper_2403_11366_amd import LoraError
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    m, n, k, r = 65536, 8192, 8192, 64
    assert lora.lora_linear_bwd_workspace_size(m, n, k, r) > lora.NOALLOC_SCRATCH_BYTES
    lib = lora.load_library()
    # validation rejects the size before any pointer is used or anything is launched
    p = [(1 << 40) + i * (1 << 36) for i in range(9)]
    assert lib.lora_linear_bwd_noalloc(*p, m, n, k, r, 128.0, None) == 5
