"""Shared helpers of the GPU tests: run the HIP path through the C ABI on
seeded inputs and compare it with the fp64 oracle."""
from __future__ import annotations

import numpy as np

import oracle
from lora_synth import Shape, gen_inputs

# Tolerances (relative Frobenius error against the fp64 oracle).
TOL_Y = 5e-3
TOL_DX = 5e-3
TOL_DA = 1e-2
TOL_DB = 1e-2
TOL_U = 1e-5     # U is an fp32 output accumulated from exact bf16 products


def rel(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    nr = np.linalg.norm(ref)
    if nr == 0.0:
        return 0.0 if np.linalg.norm(got) == 0.0 else float("inf")
    return float(np.linalg.norm(got - ref) / nr)


def f64(bits):
    return oracle.bf16_bits_to_f64(bits)


def run_gpu(t: dict, shape: Shape, poison: bool = True, stream=None, fused: bool = False):
    """Run fwd then bwd on the device (lora_linear_bwd, or lora_linear_bwd_fused
    with fused=True); returns host copies of every output."""
    import torch
    import paper_2403_11366_amd as lora
    from paper_2403_11366_amd.device_io import bits_to_device, device_to_bits

    m, n, k, r = shape.m, shape.n, shape.k, shape.r
    d = {key: bits_to_device(v) for key, v in t.items()}
    Y = torch.empty((m, n), dtype=torch.bfloat16, device="cuda")
    U = torch.empty((m, r), dtype=torch.float32, device="cuda")
    dX = torch.empty((m, k), dtype=torch.bfloat16, device="cuda")
    dA = torch.empty((r, k), dtype=torch.float32, device="cuda")
    dB = torch.empty((n, r), dtype=torch.float32, device="cuda")
    ws_size = (lora.lora_linear_bwd_fused_workspace_size if fused else lora.lora_linear_bwd_workspace_size)
    ws = torch.empty(ws_size(m, n, k, r), dtype=torch.uint8, device="cuda")
    if poison:
        for x in (Y, U, dX, dA, dB):
            x.fill_(float("nan"))
        ws.fill_(0xFF)  # bf16/fp32 NaN patterns everywhere in the workspace
    lora.lora_linear_fwd(d["X"], d["W"], d["A"], d["B"], Y, U, shape.alpha, stream=stream)
    bwd = lora.lora_linear_bwd_fused if fused else lora.lora_linear_bwd
    bwd(d["dY"], d["X"], d["W"], d["A"], d["B"], U, dX, dA, dB, ws, shape.alpha, stream=stream)
    torch.cuda.synchronize()
    return {"Y": device_to_bits(Y), "U": U.cpu().numpy(), "dX": device_to_bits(dX),
            "dA": dA.cpu().numpy(), "dB": dB.cpu().numpy()}


def sample_rows(m: int, seed: int, count: int = 48):
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 15, 16, 17, 63, 64, 127, 128, 129, 255, 256, 257, m // 2, m - 2, m - 1]
    rows = set(x for x in fixed if 0 <= x < m)
    rows |= set(rng.choice(m, size=min(count, m), replace=False).tolist())
    return sorted(rows)


def compare(t: dict, shape: Shape, out: dict, rows=None) -> dict:
    """Relative errors of every output against the oracle (Y and dX on `rows`
    only when given; U, dA and dB always whole)."""
    m = shape.m
    idx = np.arange(m) if rows is None else np.asarray(rows)
    _, Y_ref = oracle.lora_forward_rows(t["X"], t["W"], t["A"], t["B"], shape.alpha, idx)
    U_full = oracle.lora_rank_activation(t["X"], t["A"])
    dU, dX_ref, dA_ref, dB_ref = oracle.lora_backward_rows(t["dY"], t["X"], t["W"], t["A"], t["B"],
                                                          shape.alpha, idx)
    errs = {
        "Y": rel(f64(out["Y"])[idx], Y_ref),
        "U": rel(out["U"], U_full),
        "dX": rel(f64(out["dX"])[idx], dX_ref),
        "dA": rel(out["dA"], dA_ref),
        "dB": rel(out["dB"], dB_ref),
    }
    return errs


def assert_within(errs: dict, label: str = ""):
    bad = {k: v for k, v in errs.items()
           if not (v <= {"Y": TOL_Y, "U": TOL_U, "dX": TOL_DX, "dA": TOL_DA, "dB": TOL_DB}[k])}
    assert not bad, f"{label} errors over tolerance: {bad} (all: {errs})"
