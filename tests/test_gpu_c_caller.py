"""The C ABI from a program with no Python and no PyTorch
(tests/c_caller/lora_caller.cpp, built by __graft_entry__.build()): it takes
its device memory from the HIP runtime, runs lora_linear_fwd and
lora_linear_bwd, and writes the outputs back; they must match the fp64 oracle
within the stated tolerances, for a ragged shape (U pass at rank 40, ragged
tails) and the 7B q_proj shape."""
import os
import subprocess

import numpy as np
import pytest

from lora_synth import Shape, gen_inputs
from gpu_harness import assert_within, compare

pytestmark = pytest.mark.gpu

CALLER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_caller", "lora_caller")


@pytest.mark.parametrize("shape", [Shape("ccall", 300, 520, 264, 40, 80.0, 81),
                                   Shape("ccall_q", 2048, 4096, 4096, 8, 16.0, 82)],
                         ids=lambda s: f"m{s.m}n{s.n}k{s.k}r{s.r}")
def test_c_program_matches_oracle(shape, tmp_path):
    if not os.path.exists(CALLER):
        pytest.skip("tests/c_caller/lora_caller is not built (run __graft_entry__.build())")
    t = gen_inputs(shape, b_std=0.5)
    for name in ("X", "W", "A", "B", "dY"):
        np.ascontiguousarray(t[name], dtype=np.uint16).tofile(tmp_path / f"{name}.bin")
    print(f"c caller {shape}", flush=True)
    res = subprocess.run([CALLER, str(tmp_path), str(shape.m), str(shape.n), str(shape.k), str(shape.r),
                          repr(shape.alpha)], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, (res.returncode, res.stdout, res.stderr)
    m, n, k, r = shape.m, shape.n, shape.k, shape.r
    out = {"Y": np.fromfile(tmp_path / "Y.bin", dtype=np.uint16).reshape(m, n),
           "dX": np.fromfile(tmp_path / "dX.bin", dtype=np.uint16).reshape(m, k),
           "U": np.fromfile(tmp_path / "U.bin", dtype=np.float32).reshape(m, r),
           "dA": np.fromfile(tmp_path / "dA.bin", dtype=np.float32).reshape(r, k),
           "dB": np.fromfile(tmp_path / "dB.bin", dtype=np.float32).reshape(n, r)}
    assert_within(compare(t, shape, out), str(shape))
