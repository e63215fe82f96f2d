"""LoRA-adapted linear layer (JORA, arXiv 2403.11366, Eq. 1) for AMD MI355X.

Thin Python binding of the C ABI in include/lora_linear.h.  It only marshals
arguments: every step of the computation runs in the HIP kernels of
liblora_linear.so (built in-tree by ``python -m paper_2403_11366_amd.build``).
Tensors are torch device tensors (torch is used for device memory and
streams); bf16 matrices are passed as their raw 16-bit patterns.

If the library has not been built, every call raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

__all__ = [
    "LoraError", "lib_path", "load_library", "lora_linear_fwd", "lora_linear_bwd",
    "lora_linear_bwd_workspace_size", "lora_linear_bwd_noalloc", "NOALLOC_SCRATCH_BYTES", "lora_linear_bwd_fused", "lora_linear_bwd_fused_workspace_size",
    "lora_linear_merge", "lora_linear_fwd_dropout", "lora_linear_bwd_dropout",
    "lora_linear_group_fwd", "lora_linear_group_bwd", "lora_linear_group_bwd_workspace_size",
    "lora_status_string", "STATUS", "lora_linear_plan", "OPS",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "liblora_linear.so"
_lib = None

OPS = {"fwd": 0, "fwd_dropout": 1, "bwd": 2, "bwd_dropout": 3, "bwd_fused": 4, "merge": 5,
       "group_fwd": 6, "group_bwd": 7, "keep_mask": 8}

STATUS = {0: "LORA_OK", 1: "LORA_ERR_NULL", 2: "LORA_ERR_SHAPE", 3: "LORA_ERR_ALIGN",
          4: "LORA_ERR_UNSUPPORTED", 5: "LORA_ERR_WORKSPACE", 6: "LORA_ERR_ALIAS", 7: "LORA_ERR_HIP"}


class LoraError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} ({lora_status_string(status)})")


class _LaunchInfo(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_char * 128), ("grid", ctypes.c_int64), ("block", ctypes.c_int32),
                ("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32), ("member", ctypes.c_int32),
                ("col_begin", ctypes.c_int64), ("col_end", ctypes.c_int64)]


def lib_path() -> str:
    return os.path.join(_HERE, _LIB_NAME)


def load_library() -> ctypes.CDLL:
    """Load liblora_linear.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    path = lib_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2403_11366_amd.build`")
    lib = ctypes.CDLL(path)
    p, i64, f32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    lib.lora_linear_fwd.argtypes = [p, p, p, p, p, p, i64, i64, i64, i64, f32, p]
    lib.lora_linear_fwd.restype = ctypes.c_int
    lib.lora_linear_bwd_workspace_size.argtypes = [i64, i64, i64, i64]
    lib.lora_linear_bwd_workspace_size.restype = sz
    lib.lora_linear_bwd.argtypes = [p, p, p, p, p, p, p, p, p, p, sz, i64, i64, i64, i64, f32, p]
    lib.lora_linear_bwd.restype = ctypes.c_int
    lib.lora_linear_bwd_noalloc.argtypes = [p, p, p, p, p, p, p, p, p, i64, i64, i64, i64, f32, p]
    lib.lora_linear_bwd_noalloc.restype = ctypes.c_int
    lib.lora_linear_bwd_fused_workspace_size.argtypes = [i64, i64, i64, i64]
    lib.lora_linear_bwd_fused_workspace_size.restype = sz
    lib.lora_linear_bwd_fused.argtypes = [p, p, p, p, p, p, p, p, p, p, sz, i64, i64, i64, i64, f32, p]
    lib.lora_linear_bwd_fused.restype = ctypes.c_int
    lib.lora_linear_fwd_dropout.argtypes = [p, p, p, p, p, f32, p, p, i64, i64, i64, i64, f32, p]
    lib.lora_linear_fwd_dropout.restype = ctypes.c_int
    u64 = ctypes.c_uint64
    lib.lora_dropout_keep_mask.argtypes = [u64, u64, f32, p, i64, i64, p]
    lib.lora_dropout_keep_mask.restype = ctypes.c_int
    lib.lora_linear_bwd_dropout.argtypes = [p, p, p, p, p, p, p, f32, p, p, p, p, sz, i64, i64, i64, i64, f32, p]
    lib.lora_linear_bwd_dropout.restype = ctypes.c_int
    lib.lora_linear_merge.argtypes = [p, p, p, p, i64, i64, i64, f32, ctypes.c_int, p]
    lib.lora_linear_merge.restype = ctypes.c_int
    pa = ctypes.POINTER(ctypes.c_void_p)
    pn = ctypes.POINTER(ctypes.c_int64)
    lib.lora_linear_group_fwd.argtypes = [p, i64, pn, pa, pa, pa, pa, pa, i64, i64, i64, f32, p]
    lib.lora_linear_group_fwd.restype = ctypes.c_int
    lib.lora_linear_group_bwd_workspace_size.argtypes = [i64, pn, i64, i64, i64]
    lib.lora_linear_group_bwd_workspace_size.restype = sz
    lib.lora_linear_group_bwd.argtypes = [pa, p, i64, pn, pa, pa, pa, pa, p, pa, pa, p, sz, i64, i64, i64, f32, p]
    lib.lora_linear_group_bwd.restype = ctypes.c_int
    lib.lora_linear_plan.argtypes = [ctypes.c_int, i64, pn, i64, i64, i64, ctypes.POINTER(_LaunchInfo), i64]
    lib.lora_linear_plan.restype = i64
    lib.lora_status_string.argtypes = [ctypes.c_int]
    lib.lora_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def lora_status_string(status: int) -> str:
    return load_library().lora_status_string(int(status)).decode()


def lora_linear_bwd_workspace_size(m: int, n: int, k: int, r: int) -> int:
    return int(load_library().lora_linear_bwd_workspace_size(m, n, k, r))


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream_handle(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(t, name, dtype, shape):
    import torch
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous (row-major)")
    if t.device.type != "cuda":
        raise ValueError(f"{name}: must be a device tensor")
    return torch


def lora_linear_fwd(X, W, A, B, Y, U, alpha: float, stream=None) -> None:
    """Y = X W^T + (alpha/r) (X A^T) B^T and U = X A^T (see include/lora_linear.h).

    X [m,k], W [n,k], A [r,k], B [n,r], Y [m,n]: torch.bfloat16; U [m,r]: torch.float32."""
    import torch
    m, k = X.shape
    n, r = W.shape[0], A.shape[0]
    for t, name, dt, shp in ((X, "X", torch.bfloat16, (m, k)), (W, "W", torch.bfloat16, (n, k)),
                             (A, "A", torch.bfloat16, (r, k)), (B, "B", torch.bfloat16, (n, r)),
                             (Y, "Y", torch.bfloat16, (m, n)), (U, "U", torch.float32, (m, r))):
        _check(t, name, dt, shp)
    st = load_library().lora_linear_fwd(_ptr(X), _ptr(W), _ptr(A), _ptr(B), _ptr(Y), _ptr(U),
                                        m, n, k, r, float(alpha), _stream_handle(stream))
    if st != 0:
        raise LoraError(st, "lora_linear_fwd")


def lora_linear_bwd_fused_workspace_size(m: int, n: int, k: int, r: int) -> int:
    return int(load_library().lora_linear_bwd_fused_workspace_size(m, n, k, r))


def lora_linear_bwd(dY, X, W, A, B, U, dX, dA, dB, workspace, alpha: float, stream=None) -> None:
    """dX = dY W + dU A, dA = dU^T X, dB = s dY^T U with dU = s dY B, s = alpha/r.

    dY [m,n], X [m,k], W [n,k], A [r,k], B [n,r], dX [m,k]: torch.bfloat16;
    U [m,r], dA [r,k], dB [n,r]: torch.float32; workspace: a device tensor of at
    least lora_linear_bwd_workspace_size(m, n, k, r) bytes."""
    _bwd_call("lora_linear_bwd", dY, X, W, A, B, U, dX, dA, dB, workspace, alpha, stream)


NOALLOC_SCRATCH_BYTES = 32 << 20   # LORA_NOALLOC_SCRATCH_BYTES of include/lora_linear.h


def lora_linear_bwd_noalloc(dY, X, W, A, B, U, dX, dA, dB, alpha: float, stream=None) -> None:
    """lora_linear_bwd with the library's own per-GPU scratch array as the
    workspace (no allocation; calls that overlap on one GPU race on it)."""
    import torch
    m, n = dY.shape
    k, r = X.shape[1], A.shape[0]
    for t, name, dt, shp in ((dY, "dY", torch.bfloat16, (m, n)), (X, "X", torch.bfloat16, (m, k)),
                             (W, "W", torch.bfloat16, (n, k)), (A, "A", torch.bfloat16, (r, k)),
                             (B, "B", torch.bfloat16, (n, r)), (U, "U", torch.float32, (m, r)),
                             (dX, "dX", torch.bfloat16, (m, k)), (dA, "dA", torch.float32, (r, k)),
                             (dB, "dB", torch.float32, (n, r))):
        _check(t, name, dt, shp)
    st = load_library().lora_linear_bwd_noalloc(_ptr(dY), _ptr(X), _ptr(W), _ptr(A), _ptr(B), _ptr(U),
                                                _ptr(dX), _ptr(dA), _ptr(dB), m, n, k, r, float(alpha),
                                                _stream_handle(stream))
    if st != 0:
        raise LoraError(st, "lora_linear_bwd_noalloc")


def lora_linear_bwd_fused(dY, X, W, A, B, U, dX, dA, dB, workspace, alpha: float, stream=None) -> None:
    """lora_linear_bwd with dU and dB formed inside the dX GEMM (r <= 16); the
    workspace holds at least lora_linear_bwd_fused_workspace_size(m, n, k, r) bytes."""
    _bwd_call("lora_linear_bwd_fused", dY, X, W, A, B, U, dX, dA, dB, workspace, alpha, stream)


def _bwd_call(fn, dY, X, W, A, B, U, dX, dA, dB, workspace, alpha, stream):
    import torch
    m, n = dY.shape
    k, r = X.shape[1], A.shape[0]
    for t, name, dt, shp in ((dY, "dY", torch.bfloat16, (m, n)), (X, "X", torch.bfloat16, (m, k)),
                             (W, "W", torch.bfloat16, (n, k)), (A, "A", torch.bfloat16, (r, k)),
                             (B, "B", torch.bfloat16, (n, r)), (U, "U", torch.float32, (m, r)),
                             (dX, "dX", torch.bfloat16, (m, k)), (dA, "dA", torch.float32, (r, k)),
                             (dB, "dB", torch.float32, (n, r))):
        _check(t, name, dt, shp)
    if workspace.device.type != "cuda" or not workspace.is_contiguous():
        raise ValueError("workspace: must be a contiguous device tensor")
    ws_bytes = workspace.numel() * workspace.element_size()
    st = getattr(load_library(), fn)(_ptr(dY), _ptr(X), _ptr(W), _ptr(A), _ptr(B), _ptr(U),
                                     _ptr(dX), _ptr(dA), _ptr(dB), _ptr(workspace), ws_bytes,
                                     m, n, k, r, float(alpha), _stream_handle(stream))
    if st != 0:
        raise LoraError(st, fn)


def lora_linear_merge(W, A, B, W_out, alpha: float, sign: int = 1, stream=None) -> None:
    """W_out = W + sign (alpha/r) B A, rounded to bf16 (sign +1 merges, -1 unmerges).

    W, W_out [n,k], A [r,k], B [n,r]: torch.bfloat16.  W_out may be W itself."""
    import torch
    n, k = W.shape
    r = A.shape[0]
    for t, name, dt, shp in ((W, "W", torch.bfloat16, (n, k)), (A, "A", torch.bfloat16, (r, k)),
                             (B, "B", torch.bfloat16, (n, r)), (W_out, "W_out", torch.bfloat16, (n, k))):
        _check(t, name, dt, shp)
    st = load_library().lora_linear_merge(_ptr(W), _ptr(A), _ptr(B), _ptr(W_out), n, k, r, float(alpha),
                                          int(sign), _stream_handle(stream))
    if st != 0:
        raise LoraError(st, "lora_linear_merge")


def _check_keep(keep, m, k):
    import torch
    if keep.dtype != torch.uint8 or tuple(keep.shape) != (m, k // 8) or not keep.is_contiguous() \
            or keep.device.type != "cuda":
        raise ValueError(f"keep: expected a contiguous uint8 device tensor of shape {(m, k // 8)}")


def lora_dropout_keep_mask(seed: int, offset: int, p: float, keep, stream=None) -> None:
    """Draw the dropout keep mask on the device (Philox4x64-10, key (seed, 0),
    counters offset .. offset + keep.numel() - 1; see include/lora_linear.h).
    keep: contiguous uint8 device tensor [m, k/8], written."""
    import torch
    if keep.dtype != torch.uint8 or keep.dim() != 2 or not keep.is_contiguous() or keep.device.type != "cuda":
        raise ValueError("keep: expected a contiguous uint8 device tensor [m, k/8]")
    m, k = keep.shape[0], keep.shape[1] * 8
    st = load_library().lora_dropout_keep_mask(int(seed), int(offset), float(p), _ptr(keep), m, k,
                                               _stream_handle(stream))
    if st != 0:
        raise LoraError(st, "lora_dropout_keep_mask")


def lora_linear_fwd_dropout(X, W, A, B, keep, p: float, Y, U, alpha: float, stream=None) -> None:
    """Forward with dropout on the adapter input: D = keep * X / (1 - p),
    U = D A^T, Y = X W^T + (alpha/r) U B^T.  keep: uint8 [m, k/8] packed bits
    (bit l % 8 of byte l // 8 keeps element l)."""
    import torch
    m, k = X.shape
    n, r = W.shape[0], A.shape[0]
    for t, name, dt, shp in ((X, "X", torch.bfloat16, (m, k)), (W, "W", torch.bfloat16, (n, k)),
                             (A, "A", torch.bfloat16, (r, k)), (B, "B", torch.bfloat16, (n, r)),
                             (Y, "Y", torch.bfloat16, (m, n)), (U, "U", torch.float32, (m, r))):
        _check(t, name, dt, shp)
    _check_keep(keep, m, k)
    st = load_library().lora_linear_fwd_dropout(_ptr(X), _ptr(W), _ptr(A), _ptr(B), _ptr(keep), float(p), _ptr(Y),
                                                _ptr(U), m, n, k, r, float(alpha), _stream_handle(stream))
    if st != 0:
        raise LoraError(st, "lora_linear_fwd_dropout")


def lora_linear_bwd_dropout(dY, X, W, A, B, U, keep, p: float, dX, dA, dB, workspace, alpha: float,
                            stream=None) -> None:
    """Backward of lora_linear_fwd_dropout for the same keep mask and rate p."""
    import torch
    m, n = dY.shape
    k, r = X.shape[1], A.shape[0]
    for t, name, dt, shp in ((dY, "dY", torch.bfloat16, (m, n)), (X, "X", torch.bfloat16, (m, k)),
                             (W, "W", torch.bfloat16, (n, k)), (A, "A", torch.bfloat16, (r, k)),
                             (B, "B", torch.bfloat16, (n, r)), (U, "U", torch.float32, (m, r)),
                             (dX, "dX", torch.bfloat16, (m, k)), (dA, "dA", torch.float32, (r, k)),
                             (dB, "dB", torch.float32, (n, r))):
        _check(t, name, dt, shp)
    _check_keep(keep, m, k)
    if workspace.device.type != "cuda" or not workspace.is_contiguous():
        raise ValueError("workspace: must be a contiguous device tensor")
    ws_bytes = workspace.numel() * workspace.element_size()
    st = load_library().lora_linear_bwd_dropout(_ptr(dY), _ptr(X), _ptr(W), _ptr(A), _ptr(B), _ptr(U), _ptr(keep),
                                                float(p), _ptr(dX), _ptr(dA), _ptr(dB), _ptr(workspace), ws_bytes,
                                                m, n, k, r, float(alpha), _stream_handle(stream))
    if st != 0:
        raise LoraError(st, "lora_linear_bwd_dropout")


def _ptr_array(ts):
    return (ctypes.c_void_p * len(ts))(*[_ptr(t) for t in ts])


def _n_array(ns):
    return (ctypes.c_int64 * len(ns))(*[int(n) for n in ns])


def lora_linear_group_bwd_workspace_size(ns, m: int, k: int, r: int) -> int:
    return int(load_library().lora_linear_group_bwd_workspace_size(len(ns), _n_array(ns), m, k, r))


def lora_linear_group_fwd(X, Ws, As, Bs, Ys, Us, alpha: float, stream=None) -> None:
    """Projections g that read one X: U_g = X A_g^T, Y_g = X W_g^T + (alpha/r) U_g B_g^T,
    in one launch.  X [m,k], W_g [n_g,k], A_g [r,k], B_g [n_g,r], Y_g [m,n_g]:
    torch.bfloat16; U_g [m,r]: torch.float32."""
    import torch
    m, k = X.shape
    r = As[0].shape[0]
    ns = [W.shape[0] for W in Ws]
    if not (len(Ws) == len(As) == len(Bs) == len(Ys) == len(Us)):
        raise ValueError("group: W, A, B, Y, U lists must have the same length")
    _check(X, "X", torch.bfloat16, (m, k))
    for g, n in enumerate(ns):
        for t, name, dt, shp in ((Ws[g], "W", torch.bfloat16, (n, k)), (As[g], "A", torch.bfloat16, (r, k)),
                                 (Bs[g], "B", torch.bfloat16, (n, r)), (Ys[g], "Y", torch.bfloat16, (m, n)),
                                 (Us[g], "U", torch.float32, (m, r))):
            _check(t, f"{name}[{g}]", dt, shp)
    st = load_library().lora_linear_group_fwd(_ptr(X), len(ns), _n_array(ns), _ptr_array(Ws), _ptr_array(As),
                                              _ptr_array(Bs), _ptr_array(Ys), _ptr_array(Us), m, k, r,
                                              float(alpha), _stream_handle(stream))
    if st != 0:
        raise LoraError(st, "lora_linear_group_fwd")


def lora_linear_group_bwd(dYs, X, Ws, As, Bs, Us, dX, dAs, dBs, workspace, alpha: float, stream=None) -> None:
    """Backward of lora_linear_group_fwd: dX = sum_g (dY_g W_g + dU_g A_g),
    dA_g = dU_g^T X, dB_g = s dY_g^T U_g with dU_g = s dY_g B_g.  workspace: a
    device tensor of at least lora_linear_group_bwd_workspace_size(n, m, k, r) bytes."""
    import torch
    m, k = X.shape
    r = As[0].shape[0]
    ns = [W.shape[0] for W in Ws]
    if not (len(dYs) == len(Ws) == len(As) == len(Bs) == len(Us) == len(dAs) == len(dBs)):
        raise ValueError("group: dY, W, A, B, U, dA, dB lists must have the same length")
    _check(X, "X", torch.bfloat16, (m, k))
    _check(dX, "dX", torch.bfloat16, (m, k))
    for g, n in enumerate(ns):
        for t, name, dt, shp in ((dYs[g], "dY", torch.bfloat16, (m, n)), (Ws[g], "W", torch.bfloat16, (n, k)),
                                 (As[g], "A", torch.bfloat16, (r, k)), (Bs[g], "B", torch.bfloat16, (n, r)),
                                 (Us[g], "U", torch.float32, (m, r)), (dAs[g], "dA", torch.float32, (r, k)),
                                 (dBs[g], "dB", torch.float32, (n, r))):
            _check(t, f"{name}[{g}]", dt, shp)
    if workspace.device.type != "cuda" or not workspace.is_contiguous():
        raise ValueError("workspace: must be a contiguous device tensor")
    ws_bytes = workspace.numel() * workspace.element_size()
    st = load_library().lora_linear_group_bwd(_ptr_array(dYs), _ptr(X), len(ns), _n_array(ns), _ptr_array(Ws),
                                              _ptr_array(As), _ptr_array(Bs), _ptr_array(Us), _ptr(dX),
                                              _ptr_array(dAs), _ptr_array(dBs), _ptr(workspace), ws_bytes,
                                              m, k, r, float(alpha), _stream_handle(stream))
    if st != 0:
        raise LoraError(st, "lora_linear_group_bwd")


def lora_linear_plan(op: str, m: int, n, k: int, r: int) -> list:
    """The kernels the entry point `op` (a key of OPS) launches for these shapes,
    in order, as dicts (kernel name as profilers print it, grid, block, GEMM
    tile and column range, grouped member).  `n` is an int, or a list of
    output widths for the grouped ops.  Host only; raises LoraError on shapes
    the entry point would refuse."""
    ns = [int(n)] if isinstance(n, int) else [int(x) for x in n]
    lib = load_library()
    cap = 32
    buf = (_LaunchInfo * cap)()
    cnt = lib.lora_linear_plan(OPS[op], len(ns), _n_array(ns), m, k, r, buf, cap)
    if cnt < 0:
        raise LoraError(int(-cnt), f"lora_linear_plan({op})")
    return [{"kernel": buf[i].kernel.decode(), "grid": buf[i].grid, "block": buf[i].block,
             "tile": (buf[i].tile_m, buf[i].tile_n), "member": buf[i].member,
             "cols": (buf[i].col_begin, buf[i].col_end)} for i in range(min(cnt, cap))]
