"""Host-side logic that needs no GPU: the launch plans the library reports
(lora_linear_plan, the plan its entry points execute) for every shape of the
parity suites, and properties of the suites themselves."""
import pytest

from lora_synth import CONFIGS
from test_gpu_parity import DEPTH, EXACT, FULL, RAGGED, SPLIT_EDGE
from test_gpu_dropout import SHAPES as DROP_SHAPES
from test_gpu_group import CASES as GROUP_CASES, EXACT_CASES as GROUP_EXACT, FULL_GROUPS


@pytest.fixture(scope="module")
def lora():
    import paper_2403_11366_amd as lora
    try:
        lora.load_library()
    except (RuntimeError, OSError) as e:
        pytest.skip(f"library not built: {e}")
    return lora


def _gemms(plan):
    return [x for x in plan if x["tile"] != (0, 0)]


def _check_columns(gemm_launches, N):
    """The GEMM launches of a call cover output columns [0, N) once, in order,
    each with whole tiles except at the end."""
    pos = 0
    for x in gemm_launches:
        a, b = x["cols"]
        assert a == pos and b > a, (x, pos)
        assert x["grid"] >= 1
        pos = b
    assert pos == N, (gemm_launches, N)


SINGLE = RAGGED + FULL + EXACT + DEPTH + SPLIT_EDGE


@pytest.mark.parametrize("s", SINGLE, ids=lambda s: f"{s.name}-m{s.m}n{s.n}k{s.k}r{s.r}")
def test_single_projection_plans(lora, s):
    fwd = lora.lora_linear_plan("fwd", s.m, s.n, s.k, s.r)
    bwd = lora.lora_linear_plan("bwd", s.m, s.n, s.k, s.r)
    _check_columns(_gemms(fwd), s.n)
    _check_columns([x for x in bwd if "dx_kernel" in x["kernel"]], s.k)
    names = [x["kernel"] for x in bwd]
    assert names[0].startswith("lora::lora_bwd_du_dma_kernel<" if s.r % 8 == 0 else "lora::lora_bwd_du_kernel<")
    assert names[1].startswith("lora::lora_tokred_dma_kernel<")
    # the U pass precedes the first forward GEMM exactly when the rank is above
    # 16 or that GEMM is the 256 x 256 tile
    assert any("lora_u_kernel" in x["kernel"] for x in fwd) == (s.r > 16 or _gemms(fwd)[0]["tile"] == (256, 256))
    for x in bwd:
        if "dx_kernel<256, 256" in x["kernel"]:   # the 256 x 256 dX tile runs only with whole stages
            assert x["kernel"].endswith("true>"), x
        if "dx_kernel" in x["kernel"]:
            tm = -(-s.m // x["tile"][0])
            tn = -(-(x["cols"][1] - x["cols"][0]) // x["tile"][1])
            assert x["grid"] == tm * tn


def test_exact_shapes_cover_every_tile(lora):
    fwd = {x["tile"] for s in EXACT for x in _gemms(lora.lora_linear_plan("fwd", s.m, s.n, s.k, s.r))}
    dx = {x["tile"] for s in EXACT for x in lora.lora_linear_plan("bwd", s.m, s.n, s.k, s.r) if x["tile"] != (0, 0)}
    assert fwd == dx == {(256, 256), (128, 256), (128, 128)}, (fwd, dx)


def test_bench_workload_kernels(lora):
    """The 7B q_proj step is the k-split forward copying its stages straight
    into LDS, and the 128 x 256 direct-to-LDS dX."""
    s = CONFIGS["llama2_7b_q_proj"][0]
    assert [x["kernel"] for x in lora.lora_linear_plan("fwd", s.m, s.n, s.k, s.r)] == \
        ["lora::lora_fwd_ks_kernel<false, true, true, false>"]
    assert lora.lora_linear_plan("bwd", s.m, s.n, s.k, s.r)[-1]["kernel"] == \
        "lora::lora_bwd_dx_kernel<128, 256, 2, 4, 16, false, false, true>"


@pytest.mark.parametrize("s", SINGLE, ids=lambda s: f"{s.name}-m{s.m}n{s.n}k{s.k}r{s.r}")
def test_dropout_forward_is_masked_u_pass_then_plain_tiles(lora, s):
    """Under dropout the forward is the U pass with the keep mask, then the
    tiles the plain forward takes (each reading U back)."""
    if s.k % 64:
        return
    plain = lora.lora_linear_plan("fwd", s.m, s.n, s.k, s.r)
    drop = lora.lora_linear_plan("fwd_dropout", s.m, s.n, s.k, s.r)
    rp = 16 if s.r <= 16 else (32 if s.r <= 32 else 64)
    assert drop[0]["kernel"].startswith(f"lora::lora_u_kernel<{rp}, ") and drop[0]["kernel"].endswith(", true>")
    assert [x["tile"] for x in _gemms(drop)] == [x["tile"] for x in _gemms(plain)]
    assert [x["cols"] for x in _gemms(drop)] == [x["cols"] for x in _gemms(plain)]
    for x in _gemms(drop):   # every GEMM of the dropout forward reads U back
        k = x["kernel"]
        assert k.endswith("true>") if "ks_kernel" in k else k.split(",")[6].strip() == "true", k


def test_dropout_suite_reaches_every_dropout_forward_variant(lora):
    seen = {x["kernel"] for s in DROP_SHAPES for x in lora.lora_linear_plan("fwd_dropout", s.m, s.n, s.k, s.r)}
    for want in ("lora::lora_u_kernel<16, 8, true>", "lora::lora_u_kernel<16, 16, true>",
                 "lora::lora_u_kernel<16, 32, true>", "lora::lora_u_kernel<32, 8, true>",
                 "lora::lora_u_kernel<32, 16, true>", "lora::lora_u_kernel<32, 32, true>",
                 "lora::lora_u_kernel<64, 8, true>", "lora::lora_u_kernel<64, 16, true>",
                 "lora::lora_u_kernel<64, 32, true>",
                 "lora::lora_fwd_ks_kernel<false, true, true, true>",
                 "lora::lora_fwd_ks_kernel<false, true, false, true>",
                 "lora::lora_fwd_kernel<256, 256, 2, 4, 16, false, true, true, true>",
                 "lora::lora_fwd_kernel<128, 128, 2, 2, 16, false, true, true, false>"):
        assert want in seen, (want, sorted(seen))


def test_parity_suites_reach_every_plain_u_pass(lora):
    seen = {x["kernel"] for s in SINGLE for x in lora.lora_linear_plan("fwd", s.m, s.n, s.k, s.r)}
    for want in ("lora::lora_u_kernel<32, 8, false>", "lora::lora_u_kernel<32, 16, false>",
                 "lora::lora_u_kernel<32, 32, false>", "lora::lora_u_kernel<64, 8, false>",
                 "lora::lora_u_kernel<64, 16, false>", "lora::lora_u_kernel<64, 32, false>"):
        assert want in seen, (want, sorted(x for x in seen if "u_kernel" in x))


def test_parity_suites_reach_every_plannable_du_and_u_pass(lora):
    """Every dU kernel and U pass a plan can name, over token counts and ranks
    that cover each choice of tokens per workgroup and padded rank, runs in a
    GPU parity case."""
    suites = {x["kernel"] for s in SINGLE for x in lora.lora_linear_plan("bwd", s.m, s.n, s.k, s.r)}
    suites |= {x["kernel"] for s in SINGLE for x in lora.lora_linear_plan("fwd", s.m, s.n, s.k, s.r)}
    suites |= {x["kernel"] for s in DROP_SHAPES for x in lora.lora_linear_plan("fwd_dropout", s.m, s.n, s.k, s.r)}
    suites |= {x["kernel"] for s in DROP_SHAPES for x in lora.lora_linear_plan("bwd_dropout", s.m, s.n, s.k, s.r)}
    plannable = set()
    for m in (7, 2048, 4096, 8200):
        for r in range(1, 65):
            plannable |= {x["kernel"] for x in lora.lora_linear_plan("bwd", m, 128, 128, r) if "du_" in x["kernel"]}
            for n in (128, 4096):   # (4096 columns: the 256 x 256 tile, which reads U from the pass)
                for op in ("fwd", "fwd_dropout"):
                    plannable |= {x["kernel"] for x in lora.lora_linear_plan(op, m, n, 128, r) if "u_kernel" in x["kernel"]}
    missing = sorted(plannable - suites)
    assert not missing, missing


def test_parity_suites_reach_every_plannable_kernel(lora):
    """Every kernel instantiation the forward and backward plans (plain and
    dropout) can name over a sweep of token counts, widths, depths and ranks
    runs in a GPU parity case."""
    suites = set()
    for s in SINGLE:
        for op in ("fwd", "bwd"):
            suites |= {x["kernel"] for x in lora.lora_linear_plan(op, s.m, s.n, s.k, s.r)}
    for s in DROP_SHAPES:
        for op in ("fwd_dropout", "bwd_dropout"):
            suites |= {x["kernel"] for x in lora.lora_linear_plan(op, s.m, s.n, s.k, s.r)}
    plannable = {}
    for m in (7, 300, 2048, 4096, 8200):
        for n in (64, 136, 1024, 4000, 4096, 5120, 11008, 13824):
            for k in (64, 72, 1024, 4096, 4104, 5120, 11008):
                for r in (1, 8, 16, 24, 33, 40, 64):
                    ops = ("fwd", "bwd") + (("fwd_dropout", "bwd_dropout") if k % 64 == 0 else ())
                    for op in ops:
                        for x in lora.lora_linear_plan(op, m, n, k, r):
                            plannable.setdefault(x["kernel"], (op, m, n, k, r))
    missing = {kname: plannable[kname] for kname in sorted(set(plannable) - suites)}
    assert not missing, missing


def test_group_suites_reach_every_plannable_kernel(lora):
    """Every kernel instantiation the grouped forward and backward plans can
    name over a sweep of token counts, depths, ranks and member widths runs in
    a GPU case (a grouped one, or for the launches of a group of one, a
    single-projection one)."""
    groups = [(ns, m, k, r) for ns, m, k, r, _ in GROUP_CASES] + [(ns, m, k, r) for m, k, ns, r in GROUP_EXACT]
    groups += list(FULL_GROUPS)
    layer = CONFIGS["llama2_13b_layer"]
    groups += [([layer[i].n for i in mem], layer[0].m, layer[0].k, layer[0].r) for mem in ([0, 1, 2], [4, 5])]
    suites = set()
    for ns, m, k, r in groups:
        for op in ("group_fwd", "group_bwd"):
            suites |= {x["kernel"] for x in lora.lora_linear_plan(op, m, ns, k, r)}
    for s in SINGLE:
        for op in ("fwd", "bwd"):
            suites |= {x["kernel"] for x in lora.lora_linear_plan(op, s.m, s.n, s.k, s.r)}
    plannable = {}
    for m in (7, 300, 2048, 4096, 8200):
        for k in (64, 72, 1024, 4096, 4104, 5120, 13824):
            for r in (1, 8, 16, 24, 33, 64):
                for ns in ([64, 64], [136, 264, 72], [4096] * 3, [5120] * 3, [13824] * 2,
                           [64, 72, 80, 88, 96, 104, 112, 120], [5120]):
                    for op in ("group_fwd", "group_bwd"):
                        for x in lora.lora_linear_plan(op, m, ns, k, r):
                            plannable.setdefault(x["kernel"], (op, m, ns, k, r))
    missing = {kname: plannable[kname] for kname in sorted(set(plannable) - suites)}
    assert not missing, missing


def test_ragged_n_avoids_the_register_staged_256_tile(lora):
    """n not a multiple of 64 on a shape whose dX would take the 256 x 256 tile:
    the 128 x 256 tile without the FULL loads serves it."""
    for r in (8, 64):
        plan = lora.lora_linear_plan("bwd", 4096, 4000, 4096, r)
        dx = [x["kernel"] for x in plan if "dx_kernel" in x["kernel"]]
        assert dx and all(k.startswith("lora::lora_bwd_dx_kernel<128, 256,") and k.endswith("false>") for k in dx), dx


def _group_dx(lora, ns, m, k, r):
    return [x["kernel"] for x in lora.lora_linear_plan("group_bwd", m, ns, k, r) if "dx_kernel" in x["kernel"]]


def test_group_suites_reach_every_grouped_dx_variant(lora):
    """Every grouped dX variant a plan can name for these suites is run by a
    GPU test, including the 128 x 256 direct-to-LDS one (7B q/k/v)."""
    seen = set()
    for ns, m, k, r, _ in GROUP_CASES:
        seen |= set(_group_dx(lora, ns, m, k, r))
    for m, k, ns, r in GROUP_EXACT:
        seen |= set(_group_dx(lora, ns, m, k, r))
    for ns, m, k, r in FULL_GROUPS:
        seen |= set(_group_dx(lora, ns, m, k, r))
    for want in ("lora::lora_bwd_dx_kernel<128, 256, 2, 4, 16, false, true, true>",
                 "lora::lora_bwd_dx_kernel<256, 256, 2, 4, 16, false, true, true>",
                 "lora::lora_bwd_dx_kernel<128, 128, 2, 2, 16, false, true, true>"):
        assert want in seen, (want, sorted(seen))


def test_plan_refuses_what_the_entry_point_refuses(lora):
    from paper_2403_11366_amd import LoraError
    with pytest.raises(LoraError):
        lora.lora_linear_plan("fwd", 16, 100, 64, 8)        # n not a multiple of 8
    with pytest.raises(LoraError):
        lora.lora_linear_plan("bwd", 16, 64, 64, 65)        # r > 64
    with pytest.raises(LoraError):
        lora.lora_linear_plan("bwd_fused", 16, 64, 64, 32)  # fused: r <= 16
    with pytest.raises(LoraError):
        lora.lora_linear_plan("fwd_dropout", 16, 64, 72, 8)  # dropout: k % 64 == 0


def test_ragged_shapes_have_tails():
    assert any(s.m % 64 for s in RAGGED) and any(s.k % 64 for s in RAGGED)
    assert any(s.n % 64 for s in RAGGED) and {1, 64} <= {s.r for s in RAGGED}


def test_group_da_reductions_share_one_pass_over_x(lora):
    """Groups of three or more whose padded ranks add up to at most 64 share
    one dA token reduction (a stacked rank) after their own dB reductions;
    pairs and larger ranks keep one dA reduction per member."""
    plan = lora.lora_linear_plan("group_bwd", 4096, [5120] * 3, 5120, 8)     # 13B q, k, v
    red = [x for x in plan if "tokred" in x["kernel"]]
    assert [x["member"] for x in red] == [0, 1, 2, -1]
    assert red[-1]["kernel"] == "lora::lora_tokred_dma_kernel<48>"
    plan = lora.lora_linear_plan("group_bwd", 264, [392, 128, 520], 448, 64)  # 3 x 64 > 64: per member
    assert [x["member"] for x in plan if "tokred" in x["kernel"]] == [0, 1, 2]
    for ns, m, k, r, _ in GROUP_CASES:
        stacked = len(ns) >= 3 and len(ns) * (-(-r // 16) * 16) <= 64
        members = [x["member"] for x in lora.lora_linear_plan("group_bwd", m, ns, k, r) if "tokred" in x["kernel"]]
        assert (members[-1] == -1) == stacked, (ns, r, members)


def test_bench_prices_every_kernel_of_the_single_projection_plans(lora):
    """bench.py's algorithmic units (flops of the GEMMs, minimum bytes of the
    HBM-bound kernels) name every kernel the forward and backward plans of the
    Llama-2 shapes launch, except the dA/dB finalize (split-K partial traffic
    is not credited)."""
    import os
    import sys
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import bench
    for name in ("llama2_7b_q_proj", "llama2_7b_up_proj", "llama2_7b_down_proj", "llama2_13b_layer"):
        for s in CONFIGS[name]:
            for op in ("fwd", "bwd", "fwd_dropout", "bwd_dropout"):
                for x in lora.lora_linear_plan(op, s.m, s.n, s.k, s.r):
                    unit, amount = bench.algorithmic_units(s, x)
                    if x["kernel"] == "lora::lora_finalize_kernel":
                        assert unit is None
                    else:
                        assert unit in ("flop", "byte") and amount > 0, (op, s.name, x["kernel"])


def test_traffic_record_only_for_the_sources_it_was_taken_with(monkeypatch):
    """bench.py reports the committed HBM-traffic record of the dominant
    forward call only while the forward sources hash to the value the counter
    runs were taken with; after any change of those sources it reports none."""
    import json
    import bench
    path = bench.traffic_file("llama2_7b_shapes")
    with open(path) as f:
        rec = json.load(f)
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: rec["kernel_source_sha"])
    got = bench.measured_traffic("llama2_7b_shapes")
    assert got == pytest.approx(rec["hbm_bytes_per_launch"])
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0" * 16)
    assert bench.measured_traffic("llama2_7b_shapes") is None

