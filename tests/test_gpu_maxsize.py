"""The largest shapes the entry points accept: X, Y, dY and dX at 2^30 elements
each (2 GiB of bf16, the limit of one matrix), with 2^18 tokens, n = k = 4096
and rank 64 (the U pass, 256 x 256 tiles, split-K reductions over 2^18
tokens), plain and with LoRA dropout, through the C ABI.

The token rows repeat with period P: the seeded draws of P rows of X and dY
(and of the keep mask) are tiled on the device to 2^18 rows.  Then row i of
U, Y and dX is row i mod P of the oracle's P-row results, and dA and dB are
2^18 / P times the oracle's P-row dA and dB (exact scalings in fp64).  The
outputs are poisoned with NaN first and checked for NaN in full, so every
element must have been written; values are compared on sampled rows (the
first and last rows among them) and in full for dA and dB.
"""
import numpy as np
import pytest

import oracle
from lora_synth import Shape, gen_inputs, gen_keep_mask
from gpu_harness import TOL_DA, TOL_DB, TOL_DX, TOL_U, TOL_Y, f64, rel, sample_rows

pytestmark = pytest.mark.gpu

P = 512
M = 1 << 18
N = K = 4096
R = 64


@pytest.mark.parametrize("drop", [None, 0.05], ids=["plain", "dropout"])
def test_max_size_periodic_rows(drop):
    import torch
    import paper_2403_11366_amd as lora
    from paper_2403_11366_amd.device_io import bits_to_device, device_to_bits
    alpha = 2.0 * R
    sp = Shape("maxp", P, N, K, R, alpha, 91)
    print(f"max size m={M} n={N} k={K} r={R} dropout={drop}", flush=True)
    t = gen_inputs(sp, b_std=0.3)
    d = {key: bits_to_device(v) for key, v in t.items()}
    reps = M // P
    X = d["X"].repeat(reps, 1)
    dY = d["dY"].repeat(reps, 1)
    nan = float("nan")
    Y = torch.full((M, N), nan, dtype=torch.bfloat16, device="cuda")
    U = torch.full((M, R), nan, dtype=torch.float32, device="cuda")
    dX = torch.full((M, K), nan, dtype=torch.bfloat16, device="cuda")
    dA = torch.full((R, K), nan, dtype=torch.float32, device="cuda")
    dB = torch.full((N, R), nan, dtype=torch.float32, device="cuda")
    ws = torch.full((lora.lora_linear_bwd_workspace_size(M, N, K, R),), 0xFF, dtype=torch.uint8, device="cuda")
    if drop is None:
        lora.lora_linear_fwd(X, d["W"], d["A"], d["B"], Y, U, alpha)
        lora.lora_linear_bwd(dY, X, d["W"], d["A"], d["B"], U, dX, dA, dB, ws, alpha)
        U_p, Y_p = oracle.lora_forward(t["X"], t["W"], t["A"], t["B"], alpha)
        _, dX_p, dA_p, dB_p = oracle.lora_backward(t["dY"], t["X"], t["W"], t["A"], t["B"], alpha)
    else:
        keep_p = gen_keep_mask(P, K, drop, 93)
        keep = torch.from_numpy(np.ascontiguousarray(keep_p)).cuda().repeat(reps, 1)
        lora.lora_linear_fwd_dropout(X, d["W"], d["A"], d["B"], keep, drop, Y, U, alpha)
        lora.lora_linear_bwd_dropout(dY, X, d["W"], d["A"], d["B"], U, keep, drop, dX, dA, dB, ws, alpha)
        U_p, Y_p = oracle.lora_forward_dropout(t["X"], t["W"], t["A"], t["B"], keep_p, drop, alpha)
        _, dX_p, dA_p, dB_p = oracle.lora_backward_dropout(t["dY"], t["X"], t["W"], t["A"], t["B"], keep_p, drop,
                                                          alpha)
    torch.cuda.synchronize()
    for name, x in (("Y", Y), ("U", U), ("dX", dX), ("dA", dA), ("dB", dB)):
        assert not bool(torch.isnan(x).any()), f"{name} has unwritten (NaN) elements"
    rows = sample_rows(M, 5)
    idx = torch.tensor(rows, device="cuda")
    per = np.asarray(rows) % P
    e = {"Y": rel(f64(device_to_bits(Y.index_select(0, idx).contiguous())), Y_p[per]),
         "U": rel(U.index_select(0, idx).cpu().numpy(), U_p[per]),
         "dX": rel(f64(device_to_bits(dX.index_select(0, idx).contiguous())), dX_p[per]),
         "dA": rel(dA.cpu().numpy(), reps * dA_p),
         "dB": rel(dB.cpu().numpy(), reps * dB_p)}
    print({x: f"{v:.2e}" for x, v in e.items()}, flush=True)
    assert e["Y"] <= TOL_Y and e["U"] <= TOL_U and e["dX"] <= TOL_DX and e["dA"] <= TOL_DA and e["dB"] <= TOL_DB, e


def test_max_size_device_mask_sampled_rows():
    """The device keep mask at 2^18 x 4096 (128 MiB of mask bytes) against
    the oracle's generator on sampled rows."""
    import torch
    import paper_2403_11366_amd as lora
    seed, offset, p = 17, 2**50, 0.05
    keep = torch.full((M, K // 8), 0xA5, dtype=torch.uint8, device="cuda")
    lora.lora_dropout_keep_mask(seed, offset, p, keep)
    torch.cuda.synchronize()
    rows = sample_rows(M, 6, count=16)
    got = keep.index_select(0, torch.tensor(rows, device="cuda")).cpu().numpy()
    assert np.array_equal(got, oracle.dropout_keep_philox(seed, offset, p, M, K, rows=rows))
