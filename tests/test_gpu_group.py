"""GPU parity of the grouped entry points (projections that read one X, e.g.
q, k, v) through the C ABI against the fp64 oracle's grouped forward and
backward (per projection Y_g, U_g, dA_g, dB_g; the summed dX).

Tolerances are those of the single projection (Y, dX 5e-3; dA, dB 1e-2; U
1e-5).  Edge cases: a group of one (bit-identical to the plain entry points),
ragged widths per projection, every padded rank, the largest group (8),
groups whose dA reductions run as one pass over X (padded ranks adding up to
at most 64) and groups that keep one per member, integer inputs (bit for
bit), and the 13B layer's q/k/v and gate/up groups and the 7B q/k/v group at
full size with sampled dX rows.
"""
import numpy as np
import pytest

import oracle
from lora_synth import CONFIGS, Shape, gen_group_inputs, gen_ternary_inputs
from gpu_harness import TOL_DA, TOL_DB, TOL_DX, TOL_U, TOL_Y, f64, rel, run_gpu, sample_rows

pytestmark = pytest.mark.gpu


def run_group(t, m, k, r, alpha):
    import torch
    import paper_2403_11366_amd as lora
    from paper_2403_11366_amd.device_io import bits_to_device, device_to_bits
    ns = [w.shape[0] for w in t["W"]]
    G = len(ns)
    X = bits_to_device(t["X"])
    dev = {key: [bits_to_device(v) for v in t[key]] for key in ("W", "A", "B", "dY")}
    nan = float("nan")
    Y = [torch.full((m, n), nan, dtype=torch.bfloat16, device="cuda") for n in ns]
    U = [torch.full((m, r), nan, dtype=torch.float32, device="cuda") for _ in ns]
    dX = torch.full((m, k), nan, dtype=torch.bfloat16, device="cuda")
    dA = [torch.full((r, k), nan, dtype=torch.float32, device="cuda") for _ in ns]
    dB = [torch.full((n, r), nan, dtype=torch.float32, device="cuda") for n in ns]
    ws = torch.full((lora.lora_linear_group_bwd_workspace_size(ns, m, k, r),), 0xFF, dtype=torch.uint8,
                    device="cuda")
    lora.lora_linear_group_fwd(X, dev["W"], dev["A"], dev["B"], Y, U, alpha)
    lora.lora_linear_group_bwd(dev["dY"], X, dev["W"], dev["A"], dev["B"], U, dX, dA, dB, ws, alpha)
    torch.cuda.synchronize()
    return {"Y": [device_to_bits(y) for y in Y], "U": [u.cpu().numpy() for u in U],
            "dX": device_to_bits(dX), "dA": [a.cpu().numpy() for a in dA], "dB": [b.cpu().numpy() for b in dB]}


def check(t, alpha, out, rows=None):
    m = t["X"].shape[0]
    idx = np.arange(m) if rows is None else np.asarray(rows)
    U, Y = oracle.lora_group_forward(np.asarray(t["X"])[idx], t["W"], t["A"], t["B"], alpha)
    Ufull = [oracle.lora_rank_activation(t["X"], A) for A in t["A"]]
    _, dX, dA, dB = oracle.lora_group_backward(t["dY"], t["X"], t["W"], t["A"], t["B"], alpha, idx)
    e = {"dX": rel(f64(out["dX"])[idx], dX)}
    for g in range(len(t["W"])):
        e[f"Y{g}"] = rel(f64(out["Y"][g])[idx], Y[g])
        e[f"U{g}"] = rel(out["U"][g], Ufull[g])
        e[f"dA{g}"] = rel(out["dA"][g], dA[g])
        e[f"dB{g}"] = rel(out["dB"][g], dB[g])
    print({x: f"{v:.2e}" for x, v in e.items()}, flush=True)
    tol = {"Y": TOL_Y, "U": TOL_U, "dX": TOL_DX, "dA": TOL_DA, "dB": TOL_DB}
    bad = {x: v for x, v in e.items() if not v <= tol[x.rstrip("0123456789")]}
    assert not bad, bad


def _group(ns, m, k, r, alpha, seed, b_std=0.3):
    return gen_group_inputs([Shape(f"g{i}", m, n, k, r, alpha, seed + i) for i, n in enumerate(ns)], b_std=b_std)


CASES = [  # (ns, m, k, r, alpha)
    ([512, 512, 512], 256, 512, 8, 16.0),          # q, k, v of a small layer
    ([264, 136, 72], 200, 320, 5, 10.0),           # ragged widths, ragged tokens
    ([136, 256], 130, 192, 33, 66.0),              # padded rank 48
    ([392, 128, 520], 264, 448, 64, 128.0),        # rank 64
    ([1032, 1032], 520, 640, 16, 32.0),            # gate, up
    ([64, 72, 80, 88, 96, 104, 112, 120], 96, 136, 3, 6.0),   # the largest group
    ([1368, 1368, 1360], 2000, 1024, 8, 16.0),    # the k-split forward tile, ragged members
    ([264, 392], 2000, 5120, 8, 16.0),             # 2.5 rounds of 128x256 dX tiles
    ([264, 392], 4096, 4096, 8, 16.0),             # the 256x256 dX tile for a group
    ([264, 520, 136, 72], 300, 448, 13, 26.0),     # four members share one dA reduction (stacked rank 64)
] + [
    # the remaining grouped tiles a plan can name, at padded ranks 16 .. 64 with and without whole k stages:
    # the 128 x 128 forward and dX (few tokens), the 128 x 256 forward and k-split forward (130 tokens over
    # two 13824-wide members), the 256 x 256 forward (520 tokens), the 128 x 256 dX with and without whole n
    # stages, and the 256 x 256 dX
    (ns, m, k, r, 2.0 * r) for ns, m, k, r in (
        ([64, 64], 7, 64, 24), ([64, 64], 7, 72, 24), ([64, 64], 7, 72, 33), ([64, 64], 7, 1024, 24),
        ([64, 64], 7, 1024, 33), ([64, 64], 7, 1024, 64),
        ([13824, 13824], 130, 64, 24), ([13824, 13824], 130, 64, 33), ([13824, 13824], 130, 72, 1),
        ([13824, 13824], 130, 72, 24), ([13824, 13824], 130, 72, 33),
        ([6912, 6912], 520, 64, 24), ([6912, 6912], 520, 64, 33), ([6912, 6912], 520, 72, 1),
        ([6912, 6912], 520, 72, 24), ([6912, 6912], 520, 72, 33),
        ([64, 64], 2048, 2304, 24), ([64, 64], 2048, 2304, 33), ([64, 64], 2048, 2304, 64),
        ([136, 264, 72], 2048, 2304, 24), ([136, 264, 72], 2048, 2304, 33), ([136, 264, 72], 2048, 2304, 64),
        ([64, 64], 3000, 4096, 24), ([64, 64], 3000, 4096, 33), ([64, 64], 3000, 4096, 64))
]


@pytest.mark.parametrize("ns,m,k,r,alpha", CASES, ids=[f"G{len(c[0])}-m{c[1]}k{c[2]}r{c[3]}" for c in CASES])
def test_group_parity(ns, m, k, r, alpha):
    print(f"group ns={ns} m={m} k={k} r={r}", flush=True)
    t = _group(ns, m, k, r, alpha, 31 + r)
    check(t, alpha, run_group(t, m, k, r, alpha))


def test_group_of_one_matches_plain():
    m, n, k, r, alpha = 300, 520, 264, 12, 24.0
    shape = Shape("one", m, n, k, r, alpha, 41)
    t = _group([n], m, k, r, alpha, 41)
    got = run_group(t, m, k, r, alpha)
    plain = run_gpu({"X": t["X"], "W": t["W"][0], "A": t["A"][0], "B": t["B"][0], "dY": t["dY"][0]}, shape)
    assert np.array_equal(got["Y"][0], plain["Y"]) and np.array_equal(got["U"][0], plain["U"])
    assert np.array_equal(got["dA"][0], plain["dA"]) and np.array_equal(got["dB"][0], plain["dB"])
    assert np.array_equal(got["dX"], plain["dX"])
    check(t, alpha, got)


# (m, k, ns, r): the last plans the grouped 128 x 256 dX that copies its
# stages straight into LDS (every n a multiple of 64, whole column tiles)
# (the first and third take the one dA reduction of the whole group at
# stacked rank 48, the fourth at stacked rank 64, four members of rank 16)
EXACT_CASES = [(264, 1024, [512, 1024, 256], 8), (4096, 5120, [256, 512], 8), (2000, 2304, [256, 512, 192], 8),
               (1000, 1032, [256, 136, 384, 520], 16)]


@pytest.mark.parametrize("m,k,ns,r", EXACT_CASES,
                         ids=["m264k1024", "m4096k5120-dx-split", "m2000k2304-dx128x256", "m1000k1032-G4r16"])
def test_group_integer_exact(m, k, ns, r):
    """Sparse {-1, 0, 1} inputs and s = 2: every sum is a small integer, so
    the GPU matches the oracle bit for bit whatever the summation order."""
    alpha = 2.0 * r
    per = [gen_ternary_inputs(m, n, k, r, 50 + g, density=0.01) for g, n in enumerate(ns)]
    t = {"X": per[0]["X"], "W": [p["W"] for p in per], "A": [p["A"] for p in per],
         "B": [p["B"] for p in per], "dY": [p["dY"] for p in per]}
    U, Y = oracle.lora_group_forward(t["X"], t["W"], t["A"], t["B"], alpha)
    _, dX, dA, dB = oracle.lora_group_backward(t["dY"], t["X"], t["W"], t["A"], t["B"], alpha)
    assert np.abs(dX).max() <= 256 and max(np.abs(y).max() for y in Y) <= 256
    out = run_group(t, m, k, r, alpha)
    assert np.array_equal(out["dX"], oracle.f64_to_bf16_bits(dX))
    for g in range(len(ns)):
        assert np.array_equal(out["Y"][g], oracle.f64_to_bf16_bits(Y[g]))
        assert np.array_equal(out["U"][g].astype(np.float64), U[g])
        assert np.array_equal(out["dA"][g].astype(np.float64), dA[g])
        assert np.array_equal(out["dB"][g].astype(np.float64), dB[g])


@pytest.mark.parametrize("members", [[0, 1, 2], [4, 5]], ids=["13b_qkv", "13b_gate_up"])
def test_group_full_size_13b(members):
    shapes = [CONFIGS["llama2_13b_layer"][i] for i in members]
    s0 = shapes[0]
    print(f"group {[s.name for s in shapes]}", flush=True)
    t = gen_group_inputs(shapes)
    check(t, s0.alpha, run_group(t, s0.m, s0.k, s0.r, s0.alpha), sample_rows(s0.m, s0.seed))


# Other full-size groups (ns, m, k, r): the q, k, v projections of a Llama-2-7B
# attention block over 2048 tokens (its dX takes the grouped 128 x 256 tile
# that copies its stages straight into LDS).
FULL_GROUPS = [([4096, 4096, 4096], 2048, 4096, 8)]


@pytest.mark.parametrize("ns,m,k,r", FULL_GROUPS, ids=["7b_qkv"])
def test_group_full_size_other(ns, m, k, r):
    alpha = 2.0 * r
    print(f"group ns={ns} m={m} k={k} r={r}", flush=True)
    t = _group(ns, m, k, r, alpha, 61, b_std=0.02)
    check(t, alpha, run_group(t, m, k, r, alpha), sample_rows(m, 61))
