"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
rejects invalid calls before touching the GPU (no compute call is made here:
every call below fails validation, which runs before any HIP call)."""
import ctypes
import os
import re

import pytest

import paper_2403_11366_amd as lora

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(lora.lib_path()):
        from paper_2403_11366_amd import build
        build.build()
    return lora.load_library()


def declared_functions():
    names = set()
    inc = os.path.join(ROOT, "include")
    for f in os.listdir(inc):
        if f.endswith(".h"):
            text = open(os.path.join(inc, f)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names |= set(re.findall(r"\b(lora_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert {"lora_linear_fwd", "lora_linear_bwd", "lora_linear_bwd_workspace_size",
            "lora_status_string"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in range(8):
        assert lora.lora_status_string(code)
    assert lora.lora_status_string(99) == "unknown status"


# fake, 16-byte aligned, never dereferenced device addresses
BASE = 1 << 40


def addr(i, off=0):
    return BASE + i * (1 << 32) + off


def fwd(lib, ptrs=None, m=64, n=64, k=64, r=8, alpha=16.0):
    p = [addr(i) for i in range(6)] if ptrs is None else ptrs
    return lib.lora_linear_fwd(*p, m, n, k, r, alpha, None)


def bwd(lib, ptrs=None, ws_bytes=None, m=64, n=64, k=64, r=8, alpha=16.0):
    p = [addr(i) for i in range(10)] if ptrs is None else ptrs
    if ws_bytes is None:
        ws_bytes = lora.lora_linear_bwd_workspace_size(m, n, k, r)
    return lib.lora_linear_bwd(*p, ws_bytes, m, n, k, r, alpha, None)


def test_fwd_null(lib):
    for i in range(6):
        p = [addr(j) for j in range(6)]
        p[i] = None
        assert fwd(lib, p) == 1


@pytest.mark.parametrize("m,n,k,r,code", [(0, 64, 64, 8, 2), (64, 0, 64, 8, 2), (64, 64, 0, 8, 2),
                                          (64, 64, 64, 0, 2), (64, 60, 64, 8, 2), (64, 64, 12, 8, 2),
                                          (-1, 64, 64, 8, 2), (64, 64, 64, 65, 4),
                                          (1 << 23, 64, 64, 8, 4), (1 << 21, 1 << 20, 64, 8, 4)])
def test_fwd_bad_shapes(lib, m, n, k, r, code):
    assert fwd(lib, m=m, n=n, k=k, r=r) == code


def test_fwd_misaligned(lib):
    for i in range(6):
        p = [addr(j) for j in range(6)]
        p[i] += 8
        assert fwd(lib, p) == 3


def test_fwd_alias(lib):
    p = [addr(j) for j in range(6)]
    p[4] = p[0] + 16  # Y inside X
    assert fwd(lib, p) == 6
    p = [addr(j) for j in range(6)]
    p[5] = p[4] + 64  # U inside Y
    assert fwd(lib, p) == 6


def test_bwd_null(lib):
    for i in range(10):
        p = [addr(j) for j in range(10)]
        p[i] = None
        code = bwd(lib, p)
        assert code == (5 if i == 9 else 1)


def test_bwd_workspace(lib):
    need = lora.lora_linear_bwd_workspace_size(64, 64, 64, 8)
    assert need > 0 and need % 256 == 0
    assert bwd(lib, ws_bytes=need - 1) == 5
    assert lora.lora_linear_bwd_workspace_size(64, 60, 64, 8) == 0
    assert lora.lora_linear_bwd_workspace_size(64, 64, 64, 65) == 0


def test_bwd_misaligned_and_alias(lib):
    for i in range(10):
        p = [addr(j) for j in range(10)]
        p[i] += 4
        assert bwd(lib, p) == 3
    p = [addr(j) for j in range(10)]
    p[6] = p[0]            # dX on top of dY
    assert bwd(lib, p) == 6
    p = [addr(j) for j in range(10)]
    p[9] = p[1] + 1024     # workspace inside X
    assert bwd(lib, p) == 6
    p = [addr(j) for j in range(10)]
    p[8] = p[7] + 16       # dB inside dA
    assert bwd(lib, p) == 6


@pytest.mark.parametrize("m,n,k,r,code", [(0, 64, 64, 8, 2), (64, 64, 64, 65, 4), (64, 8, 7, 8, 2)])
def test_bwd_bad_shapes(lib, m, n, k, r, code):
    assert bwd(lib, ws_bytes=1 << 30, m=m, n=n, k=k, r=r) == code


def merge(lib, ptrs=None, n=64, k=64, r=8, alpha=16.0, sign=1):
    p = [addr(i) for i in range(4)] if ptrs is None else ptrs
    return lib.lora_linear_merge(*p, n, k, r, alpha, sign, None)


def test_merge_null_and_sign(lib):
    for i in range(4):
        p = [addr(j) for j in range(4)]
        p[i] = None
        assert merge(lib, p) == 1
    for sign in (0, 2, -2):
        assert merge(lib, sign=sign) == 2


@pytest.mark.parametrize("n,k,r,code", [(0, 64, 8, 2), (64, 60, 8, 2), (64, 64, 0, 2), (64, 64, 65, 4),
                                        (1 << 23, 64, 8, 4)])
def test_merge_bad_shapes(lib, n, k, r, code):
    assert merge(lib, n=n, k=k, r=r) == code


def test_merge_misaligned_and_alias(lib):
    for i in range(4):
        p = [addr(j) for j in range(4)]
        p[i] += 2
        assert merge(lib, p) == 3
    p = [addr(j) for j in range(4)]
    p[3] = p[0] + 16          # W_out shifted inside W (in place means exactly W)
    assert merge(lib, p) == 6
    p = [addr(j) for j in range(4)]
    p[3] = p[2]               # W_out on top of B
    assert merge(lib, p) == 6


def fwd_drop(lib, ptrs=None, p=0.05, m=64, n=64, k=64, r=8, alpha=16.0):
    q = [addr(i) for i in range(7)] if ptrs is None else ptrs
    return lib.lora_linear_fwd_dropout(q[0], q[1], q[2], q[3], q[4], p, q[5], q[6], m, n, k, r, alpha, None)


def bwd_drop(lib, ptrs=None, p=0.05, m=64, n=64, k=64, r=8, alpha=16.0, ws_bytes=None):
    q = [addr(i) for i in range(11)] if ptrs is None else ptrs
    if ws_bytes is None:
        ws_bytes = lora.lora_linear_bwd_workspace_size(m, n, k, r)
    return lib.lora_linear_bwd_dropout(q[0], q[1], q[2], q[3], q[4], q[5], q[6], p, q[7], q[8], q[9], q[10],
                                       ws_bytes, m, n, k, r, alpha, None)


def test_dropout_validation(lib):
    for i in range(7):
        q = [addr(j) for j in range(7)]
        q[i] = None
        assert fwd_drop(lib, q) == 1
    for p in (-0.1, 1.0, 2.0, float("nan")):
        assert fwd_drop(lib, p=p) == 2
        assert bwd_drop(lib, p=p) == 2
    assert fwd_drop(lib, k=72) == 2          # k must be a multiple of 64 with dropout
    assert bwd_drop(lib, k=72, ws_bytes=1 << 30) == 2
    q = [addr(j) for j in range(7)]
    q[4] += 8                                 # keep mask misaligned
    assert fwd_drop(lib, q) == 3
    q = [addr(j) for j in range(7)]
    q[5] = q[4] + 64                          # Y on top of the keep mask
    assert fwd_drop(lib, q) == 6
    q = [addr(j) for j in range(11)]
    q[6] = None
    assert bwd_drop(lib, q) == 1
    q = [addr(j) for j in range(11)]
    q[7] = q[6]                               # dX on top of the keep mask
    assert bwd_drop(lib, q) == 6


def _parr(vals):
    return (ctypes.c_void_p * len(vals))(*vals)


def _narr(vals):
    return (ctypes.c_int64 * len(vals))(*vals)


def group_fwd(lib, G=3, ns=None, m=64, k=64, r=8, X=None, arrays=None):
    ns = ns or [64] * G
    base = 1 << 44
    arr = arrays or {key: [base + (j * 16 + g) * (1 << 30) for g in range(G)] for j, key in enumerate("WABYU")}
    X = addr(40) if X is None else X
    return lib.lora_linear_group_fwd(X, G, _narr(ns), _parr(arr["W"]), _parr(arr["A"]), _parr(arr["B"]),
                                     _parr(arr["Y"]), _parr(arr["U"]), m, k, r, 16.0, None)


def group_bwd(lib, G=2, ns=None, m=64, k=64, r=8, ws_bytes=1 << 30, arrays=None, dX=None, ws=None):
    ns = ns or [64] * G
    base = 1 << 44
    arr = arrays or {key: [base + (j * 16 + g) * (1 << 30) for g in range(G)]
                     for j, key in enumerate(["dY", "W", "A", "B", "U", "dA", "dB"])}
    dX = addr(41) if dX is None else dX
    ws = addr(42) if ws is None else ws
    return lib.lora_linear_group_bwd(_parr(arr["dY"]), addr(40), G, _narr(ns), _parr(arr["W"]), _parr(arr["A"]),
                                     _parr(arr["B"]), _parr(arr["U"]), dX, _parr(arr["dA"]), _parr(arr["dB"]),
                                     ws, ws_bytes, m, k, r, 16.0, None)


def test_group_validation(lib):
    assert group_fwd(lib, G=0) == 2
    assert group_fwd(lib, G=9, ns=[64] * 9) == 4
    assert group_fwd(lib, ns=[64, 72 + 4, 64]) == 2          # n not a multiple of 8
    assert group_fwd(lib, r=65) == 4
    assert lib.lora_linear_group_fwd(addr(40), 3, None, None, None, None, None, None, 64, 64, 8, 16.0, None) == 1
    base = 1 << 44
    arr = {key: [base + (j * 16 + g) * (1 << 30) for g in range(3)] for j, key in enumerate("WABYU")}
    arr["B"][1] = 0
    assert group_fwd(lib, arrays=arr) == 1
    arr["B"][1] = base + 8                                   # misaligned
    assert group_fwd(lib, arrays=arr) == 3
    arr["B"][1] = base + (2 * 16 + 1) * (1 << 30)
    arr["Y"][2] = arr["W"][0]                                # output on an input
    assert group_fwd(lib, arrays=arr) == 6
    arr["Y"][2] = arr["U"][0]                                # two outputs overlap
    assert group_fwd(lib, arrays=arr) == 6
    assert group_fwd(lib, X=base + (3 * 16 + 0) * (1 << 30) + 64) == 6   # X inside Y[0]
    ns = [64, 128]
    need = lora.lora_linear_group_bwd_workspace_size(ns, 64, 64, 8)
    assert need >= lora.lora_linear_bwd_workspace_size(64, 64, 64, 8) + lora.lora_linear_bwd_workspace_size(64, 128, 64, 8)
    assert lora.lora_linear_group_bwd_workspace_size([64, 60], 64, 64, 8) == 0
    assert group_bwd(lib, ns=ns, ws_bytes=need - 1) == 5
    assert group_bwd(lib, ns=ns, ws=addr(42, 8)) == 3
    assert group_bwd(lib, ns=ns, dX=addr(40)) == 6           # dX on X
    arr = {key: [base + (j * 16 + g) * (1 << 30) for g in range(2)]
           for j, key in enumerate(["dY", "W", "A", "B", "U", "dA", "dB"])}
    arr["dA"][1] = arr["dB"][0]
    assert group_bwd(lib, ns=ns, arrays=arr) == 6
    arr["dA"][1] = base + (5 * 16 + 1) * (1 << 30)
    arr["dY"][0] = 0
    assert group_bwd(lib, ns=ns, arrays=arr) == 1


def bwd_fused(lib, ptrs=None, ws_bytes=None, m=64, n=64, k=64, r=8, alpha=16.0):
    p = [addr(i) for i in range(10)] if ptrs is None else ptrs
    if ws_bytes is None:
        ws_bytes = lora.lora_linear_bwd_fused_workspace_size(m, n, k, r)
    return lib.lora_linear_bwd_fused(*p, ws_bytes, m, n, k, r, alpha, None)


def test_bwd_fused_validation(lib):
    need = lora.lora_linear_bwd_fused_workspace_size(64, 64, 64, 8)
    assert need > 0 and need % 256 == 0
    assert lora.lora_linear_bwd_fused_workspace_size(64, 64, 64, 17) == 0   # rank above 16
    assert lora.lora_linear_bwd_fused_workspace_size(64, 60, 64, 8) == 0
    assert bwd_fused(lib, ws_bytes=need - 1) == 5
    assert bwd_fused(lib, ws_bytes=1 << 30, r=17) == 4
    assert bwd_fused(lib, ws_bytes=1 << 30, r=65) == 4
    assert bwd_fused(lib, ws_bytes=1 << 30, m=0) == 2
    for i in range(10):
        p = [addr(j) for j in range(10)]
        p[i] = None
        assert bwd_fused(lib, p) == (5 if i == 9 else 1)
        p = [addr(j) for j in range(10)]
        p[i] += 4
        assert bwd_fused(lib, p) == 3
    p = [addr(j) for j in range(10)]
    p[6] = p[0]            # dX on top of dY
    assert bwd_fused(lib, p) == 6
    p = [addr(j) for j in range(10)]
    p[9] = p[2] + 256      # workspace inside W
    assert bwd_fused(lib, p) == 6


def test_keep_mask_validation(lib):
    f = lib.lora_dropout_keep_mask
    assert f(1, 0, 0.05, None, 64, 64, None) == 1
    for p in (-0.1, 1.0, 2.0, float("nan")):
        assert f(1, 0, p, addr(0), 64, 64, None) == 2
    for m, k in ((0, 64), (64, 0), (64, 12), (-1, 64)):
        assert f(1, 0, 0.05, addr(0), m, k, None) == 2
    assert f(1, 0, 0.05, addr(0) + 8, 64, 64, None) == 3   # misaligned


def test_keep_mask_plan(lib):
    plan = lora.lora_linear_plan("keep_mask", 300, 64, 1024, 1)
    assert [x["kernel"] for x in plan] == ["lora::lora_keep_mask_kernel"]
    assert plan[0]["grid"] == -(-300 * 128 // (4 * 256)) and plan[0]["block"] == 256
    with pytest.raises(lora.LoraError):
        lora.lora_linear_plan("keep_mask", 300, 64, 12, 1)
