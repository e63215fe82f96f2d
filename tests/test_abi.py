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
