"""GPU parity of the LoRA-dropout entry points (through the C ABI) against the
fp64 oracle, with the keep mask drawn by the seeded input generator.

Tolerances are those of the plain path (Y, dX 5e-3; dA, dB 1e-2; U 1e-5).
Edge cases: every element kept with p = 0 (the forward and dA, dB then match
the plain entry points bit for bit), nothing kept (U, dA and dB exactly zero,
Y and dX the frozen path alone), ragged shapes and every padded rank.
"""
import numpy as np
import pytest

import oracle
from lora_synth import Shape, gen_inputs, gen_keep_mask
from gpu_harness import TOL_DA, TOL_DB, TOL_DX, TOL_U, TOL_Y, f64, rel, run_gpu

pytestmark = pytest.mark.gpu


def run_dropout(t, shape, keep, p, device_keep=None):
    import torch
    import paper_2403_11366_amd as lora
    from paper_2403_11366_amd.device_io import bits_to_device, device_to_bits
    m, n, k, r = shape.m, shape.n, shape.k, shape.r
    d = {key: bits_to_device(v) for key, v in t.items()}
    kd = torch.from_numpy(np.ascontiguousarray(keep)).cuda() if device_keep is None else device_keep
    Y = torch.full((m, n), float("nan"), dtype=torch.bfloat16, device="cuda")
    U = torch.full((m, r), float("nan"), dtype=torch.float32, device="cuda")
    dX = torch.full((m, k), float("nan"), dtype=torch.bfloat16, device="cuda")
    dA = torch.full((r, k), float("nan"), dtype=torch.float32, device="cuda")
    dB = torch.full((n, r), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.full((lora.lora_linear_bwd_workspace_size(m, n, k, r),), 0xFF, dtype=torch.uint8, device="cuda")
    lora.lora_linear_fwd_dropout(d["X"], d["W"], d["A"], d["B"], kd, p, Y, U, shape.alpha)
    lora.lora_linear_bwd_dropout(d["dY"], d["X"], d["W"], d["A"], d["B"], U, kd, p, dX, dA, dB, ws, shape.alpha)
    torch.cuda.synchronize()
    return {"Y": device_to_bits(Y), "U": U.cpu().numpy(), "dX": device_to_bits(dX),
            "dA": dA.cpu().numpy(), "dB": dB.cpu().numpy()}


def check(t, shape, keep, p, out):
    U, Y = oracle.lora_forward_dropout(t["X"], t["W"], t["A"], t["B"], keep, p, shape.alpha)
    _, dX, dA, dB = oracle.lora_backward_dropout(t["dY"], t["X"], t["W"], t["A"], t["B"], keep, p, shape.alpha)
    e = {"Y": rel(f64(out["Y"]), Y), "U": rel(out["U"], U), "dX": rel(f64(out["dX"]), dX),
         "dA": rel(out["dA"], dA), "dB": rel(out["dB"], dB)}
    print(shape, p, {x: f"{v:.2e}" for x, v in e.items()}, flush=True)
    assert e["Y"] <= TOL_Y and e["dX"] <= TOL_DX and e["dA"] <= TOL_DA and e["dB"] <= TOL_DB and e["U"] <= TOL_U
    return e


SHAPES = [Shape("drop_tiny", 256, 512, 512, 8, 16.0, 21), Shape("drop_ragged", 200, 264, 320, 5, 10.0, 22),
          Shape("drop_128x256", 2000, 4000, 1024, 5, 10.0, 28),  # the 128 x 256 tile, ragged m and n
          Shape("drop_r33", 130, 136, 192, 33, 66.0, 23), Shape("drop_r64", 264, 392, 448, 64, 128.0, 24),
          Shape("drop_r16", 520, 1032, 640, 16, 32.0, 25),
          Shape("drop_256x256", 1536, 8192, 256, 8, 16.0, 29),    # the 256 x 256 tile reading U back
          Shape("drop_ks_rounds", 2431, 6656, 256, 13, 26.0, 30),  # k-split tile over several rounds
          Shape("drop_split", 2560, 8192, 256, 13, 26.0, 39),      # 256 x 256 columns, then one k-split round
          # the masked U pass with 32 tokens per workgroup (8192 tokens and more) at padded ranks 16, 32, 64,
          # and with 16 at rank 32
          Shape("drop_m8192", 8200, 264, 256, 8, 16.0, 31), Shape("drop_m8192_r24", 8192, 136, 128, 24, 48.0, 32),
          Shape("drop_m8192_r64", 8192, 128, 192, 64, 128.0, 33), Shape("drop_r24", 300, 264, 192, 24, 48.0, 34),
          # the masked dX tiles of every padded rank: 128 x 128 at 32, 48, 64; 128 x 256 at 16 .. 64 with and
          # without whole stages (n a multiple of 64 or not)
          Shape("drop_dx128_r24", 7, 64, 1024, 24, 48.0, 40), Shape("drop_dx128_r33", 7, 64, 1024, 33, 66.0, 41),
          Shape("drop_dx128_r64", 7, 64, 1024, 64, 128.0, 42),
          Shape("drop_dx256_r1", 300, 136, 11008, 1, 2.0, 43), Shape("drop_dx256f_r1", 300, 64, 11008, 1, 2.0, 44),
          Shape("drop_dx256_r24", 300, 136, 11008, 24, 48.0, 45),
          Shape("drop_dx256f_r24", 300, 64, 11008, 24, 48.0, 46),
          Shape("drop_dx256_r33", 300, 136, 11008, 33, 66.0, 47),
          Shape("drop_dx256f_r33", 300, 64, 11008, 33, 66.0, 48),
          Shape("drop_dx256_r64", 300, 136, 11008, 64, 128.0, 49),
          Shape("drop_dx256f_r64", 300, 64, 11008, 64, 128.0, 50),
          # U pass with 16-token workgroups (4096 <= m < 8192; smaller m takes 8-token ones)
          Shape("drop_m4100", 4100, 136, 128, 8, 16.0, 51), Shape("drop_m4100_r24", 4100, 136, 128, 24, 48.0, 52),
          Shape("drop_m4096_r64", 4096, 128, 192, 64, 128.0, 53)]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: s.name)
@pytest.mark.parametrize("p", [0.05, 0.5])
def test_dropout_parity(shape, p):
    t = gen_inputs(shape, b_std=0.3)
    keep = gen_keep_mask(shape.m, shape.k, p, shape.seed + 7)
    check(t, shape, keep, p, run_dropout(t, shape, keep, p))


def test_dropout_full_size_q_proj():
    shape = Shape("llama2_7b_q_proj", 2048, 4096, 4096, 8, 16.0, 1000)
    t = gen_inputs(shape)
    keep = gen_keep_mask(shape.m, shape.k, 0.05, 31)
    check(t, shape, keep, 0.05, run_dropout(t, shape, keep, 0.05))


def test_dropout_keep_all_matches_plain_path():
    shape = Shape("drop_all_kept", 192, 256, 320, 12, 24.0, 26)
    t = gen_inputs(shape, b_std=0.3)
    keep = np.full((shape.m, shape.k // 8), 0xFF, dtype=np.uint8)
    got = run_dropout(t, shape, keep, 0.0)
    plain = run_gpu(t, shape)
    # the two paths form U (the U pass against the tile) and reduce dA and dB
    # (the masked reduction stages X through registers) with different
    # kernels, so their fp32 sums differ in order only; Y and dX then differ
    # by at most the odd flipped bf16 rounding
    for x in ("U", "dA", "dB"):
        assert rel(got[x], plain[x]) <= 1e-5, x
    for x in ("Y", "dX"):
        assert rel(f64(got[x]), f64(plain[x])) <= 1e-3, x
    check(t, shape, keep, 0.0, got)


def test_dropout_keep_none():
    shape = Shape("drop_none_kept", 136, 200, 256, 8, 16.0, 27)
    t = gen_inputs(shape, b_std=0.3)
    keep = np.zeros((shape.m, shape.k // 8), dtype=np.uint8)
    out = run_dropout(t, shape, keep, 0.3)
    assert not out["U"].any() and not out["dA"].any() and not out["dB"].any()
    check(t, shape, keep, 0.3, out)


# The keep mask drawn on the device (lora_dropout_keep_mask, Philox4x64-10)
# against the oracle's evaluation of the same generator, bit for bit: ragged
# byte counts (not a multiple of the 16 bytes a thread writes), a counter
# that carries into its second word, p = 0, and the 7B q_proj input on
# sampled rows.
MASK_CASES = [(300, 1024, 1, 0, 0.05), (37, 72, 2**64 - 1, 2**64 - 5, 0.5), (3, 24, 7, 123, 0.3),
              (1, 8, 0, 0, 0.0), (129, 4104, 42, 2**40, 0.05), (5, 40, 3, 2**64 - 2, 0.9)]


def _device_mask(seed, offset, p, m, k):
    import torch
    import paper_2403_11366_amd as lora
    keep = torch.full((m, k // 8), 0xA5, dtype=torch.uint8, device="cuda")
    lora.lora_dropout_keep_mask(seed, offset, p, keep)
    torch.cuda.synchronize()
    return keep


@pytest.mark.parametrize("m,k,seed,offset,p", MASK_CASES)
def test_device_keep_mask_matches_oracle(m, k, seed, offset, p):
    print(f"mask m={m} k={k} seed={seed} offset={offset} p={p}", flush=True)
    got = _device_mask(seed, offset, p, m, k).cpu().numpy()
    assert np.array_equal(got, oracle.dropout_keep_philox(seed, offset, p, m, k))


def test_device_keep_mask_full_size_sampled_rows():
    from gpu_harness import sample_rows
    m, k, seed, offset, p = 2048, 4096, 2024, 2**33, 0.05
    got = _device_mask(seed, offset, p, m, k).cpu().numpy()
    rows = sample_rows(m, 7)
    assert np.array_equal(got[rows], oracle.dropout_keep_philox(seed, offset, p, m, k, rows=rows))
    bits = np.unpackbits(got, bitorder="little")
    q = oracle.keep_threshold(p) / 2**16
    assert abs(bits.mean() - q) <= 5 * np.sqrt(q * (1 - q) / bits.size)


def test_dropout_step_with_device_mask():
    """A training step whose mask never leaves the device: the forward and
    backward read the generated mask, and match the oracle given the oracle's
    mask of the same (seed, offset, p)."""
    import torch
    shape = Shape("drop_dev", 520, 1032, 640, 16, 32.0, 51)
    p = 0.05
    keep = oracle.dropout_keep_philox(77, 5000, p, shape.m, shape.k)
    assert np.array_equal(_device_mask(77, 5000, p, shape.m, shape.k).cpu().numpy(), keep)
    t = gen_inputs(shape, b_std=0.5)
    check(t, shape, keep, p, run_dropout(t, shape, keep, p, device_keep=_device_mask(77, 5000, p, shape.m, shape.k)))
