"""Thin ctypes binding of the C ABI in ``include/dfa.h`` (``libdfa.so``).

Argument marshalling only: each function takes torch tensors, checks that they
are contiguous [B, H, L, d] tensors on a GPU (bf16, the residual R fp32),
reads B, H, L, d from the
shapes, and calls the C function of the same name with the tensors' device
pointers and the current HIP stream.  All computation happens in the
library's HIP kernels; there is no fallback of any kind.  A non-OK status
raises :class:`DfaError` with the library's message.

``lib()`` exposes the raw ctypes handle for callers that marshal pointers
themselves (the ABI tests do).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from .build import LIB_PATH

DFA_OK, DFA_ERR_INVALID_ARG, DFA_ERR_UNSUPPORTED, DFA_ERR_HIP = 0, 1, 2, 3
FULL, WARS_REFRESH, WARS_REUSE, AST_REUSE, ASC_REUSE = 0, 1, 2, 3, 4
WARS_ASC_REFRESH, WARS_ASC_REUSE = 5, 6
CODE_NAMES = {FULL: "FULL", WARS_REFRESH: "WARS_REFRESH", WARS_REUSE: "WARS_REUSE",
              AST_REUSE: "AST_REUSE", ASC_REUSE: "ASC_REUSE",
              WARS_ASC_REFRESH: "WARS_ASC_REFRESH", WARS_ASC_REUSE: "WARS_ASC_REUSE"}

# every symbol include/dfa.h declares
EXPORTS = ("dfa_attn_full", "dfa_attn_full_and_residual", "dfa_attn_window_plus_residual",
           "dfa_plan_step", "dfa_plan_make", "dfa_qkv_proj", "dfa_out_proj", "dfa_module_step",
           "dfa_mrae", "dfa_mrae_noalloc", "dfa_plan_search_workspace_bytes", "dfa_plan_search", "dfa_last_error", "dfa_version")
MRAE_WORKSPACE_BYTES = 8192


class DfaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"dfa status {status}: {message}")
        self.status = status


_LIB = None
_vp, _int, _i32p = ctypes.c_void_p, ctypes.c_int, ctypes.POINTER(ctypes.c_int32)


def lib() -> ctypes.CDLL:
    """Load libdfa.so (built in-tree; the environment variable DFA_LIBRARY
    names another build of the same sources); raises if it is missing."""
    global _LIB
    if _LIB is None:
        path = os.environ.get("DFA_LIBRARY") or LIB_PATH
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it first "
                               "(python -c 'import __graft_entry__ as g; g.build()')")
        L = ctypes.CDLL(path)
        attn = [_vp, _vp, _vp, _vp, _vp, _int, _int, _int, _int, _int, _vp]
        for name in ("dfa_attn_full", "dfa_attn_full_and_residual", "dfa_attn_window_plus_residual"):
            f = getattr(L, name)
            f.argtypes = attn
            f.restype = _int
        L.dfa_plan_step.argtypes = [_int, _vp, _vp, _vp, _vp, _vp, _vp, _int, _int, _int, _int, _int, _vp]
        L.dfa_plan_step.restype = _int
        L.dfa_plan_make.argtypes = [ctypes.c_uint64, _int, _int, _int, _int, _i32p, _i32p, _i32p]
        L.dfa_plan_make.restype = _int
        L.dfa_qkv_proj.argtypes = [_vp] * 6 + [_int] * 4 + [_vp]
        L.dfa_qkv_proj.restype = _int
        L.dfa_out_proj.argtypes = [_vp] * 4 + [_int] * 4 + [_vp]
        L.dfa_out_proj.restype = _int
        L.dfa_module_step.argtypes = [_int] + [_vp] * 12 + [_int] * 5 + [_vp]
        L.dfa_module_step.restype = _int
        L.dfa_mrae.argtypes = [_vp, _vp, ctypes.c_size_t, _vp, _vp, _vp]
        L.dfa_mrae.restype = _int
        L.dfa_mrae_noalloc.argtypes = [_vp, _vp, ctypes.c_size_t, _vp, _vp]
        L.dfa_mrae_noalloc.restype = _int
        L.dfa_plan_search_workspace_bytes.argtypes = [_int] * 5
        L.dfa_plan_search_workspace_bytes.restype = ctypes.c_size_t
        _vpp = ctypes.POINTER(ctypes.c_void_p)
        L.dfa_plan_search.argtypes = [_int, _int, _vpp, _vpp, _vpp, _vpp, _vpp, ctypes.c_double] + [_int] * 5 + \
            [_vp, ctypes.c_size_t, _i32p, ctypes.POINTER(ctypes.c_double), _vp]
        L.dfa_plan_search.restype = _int
        L.dfa_last_error.argtypes = []
        L.dfa_last_error.restype = ctypes.c_char_p
        L.dfa_version.argtypes = []
        L.dfa_version.restype = ctypes.c_char_p
        _LIB = L
    return _LIB


def last_error() -> str:
    return lib().dfa_last_error().decode()


def _check(status: int) -> None:
    if status != DFA_OK:
        raise DfaError(status, last_error())


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


_TORCH = None
_RAW_STREAM = None


def _torch():
    """torch, imported on first use (the ABI tests run without a GPU)."""
    global _TORCH, _RAW_STREAM
    if _TORCH is None:
        import torch
        _TORCH = torch
        _RAW_STREAM = getattr(torch._C, "_cuda_getCurrentRawStream", None)
    return _TORCH


def _shape(*tensors, R=None):
    torch = _torch()
    ref = tensors[0]
    shape = ref.shape
    bf16, f32 = torch.bfloat16, torch.float32
    for t in (*tensors, R):
        if t is None:
            continue
        want = f32 if t is R else bf16
        if t.dtype != want:
            raise TypeError(f"expected {want} (R is fp32, the rest bf16), got {t.dtype}")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous [B, H, L, d]")
        if not t.is_cuda:
            raise ValueError("tensors must live on a GPU")
        if t.shape != shape or t.dim() != 4:
            raise ValueError(f"shape mismatch: {tuple(t.shape)} vs {tuple(shape)}")
    return tuple(shape)


def _stream(stream) -> int:
    """The HIP stream handle of `stream`, or of torch's current stream.  The
    raw query returns the same handle as torch.cuda.current_stream() without
    building a Stream object (a few microseconds per call)."""
    torch = _torch()
    if stream is None:
        if _RAW_STREAM is not None:
            return _RAW_STREAM(torch.cuda.current_device())
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def dfa_attn_full(Q, K, V, O, w: int = 0, stream=None) -> None:
    """O = softmax(Q K^T / sqrt(d)) V."""
    B, H, L, d = _shape(Q, K, V, O)
    _check(lib().dfa_attn_full(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), None, B, H, L, d, w, _stream(stream)))


def dfa_attn_full_and_residual(Q, K, V, O, R, w: int, stream=None) -> None:
    """O = full attention and R (fp32) = O - window attention (|i-j| <= w)."""
    B, H, L, d = _shape(Q, K, V, O, R=R)
    _check(lib().dfa_attn_full_and_residual(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(R), B, H, L, d, w,
                                            _stream(stream)))


def dfa_attn_window_plus_residual(Q, K, V, O, R, w: int, stream=None) -> None:
    """O = window attention (|i-j| <= w) + R (fp32; None: window attention only)."""
    B, H, L, d = _shape(Q, K, V, O, R=R)
    _check(lib().dfa_attn_window_plus_residual(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(R), B, H, L, d, w,
                                               _stream(stream)))


def dfa_plan_step(code: int, Q, K, V, O, R, Ocache, w: int, stream=None) -> None:
    """One plan entry of one layer (see include/dfa.h for the cache rules)."""
    B, H, L, d = _shape(O, Q, K, V, Ocache, R=R)
    _check(lib().dfa_plan_step(int(code), _ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(R), _ptr(Ocache),
                               B, H, L, d, w, _stream(stream)))


def _expect(t, dtype, shape, name):
    if t is None:
        return
    if t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or not t.is_cuda:
        raise ValueError(f"{name}: expected a contiguous {dtype} GPU tensor of shape {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


def _proj_shapes(X, Q):
    """B, H, L, d from X [B, L, C] and a [B, H, L, d] tensor."""
    B, H, L, d = Q.shape
    if tuple(X.shape) != (B, L, H * d):
        raise ValueError(f"X {tuple(X.shape)} does not match [B, L, H*d] = {(B, L, H * d)}")
    return B, H, L, d


def _weights(Wqkv, bqkv, Wo, bo, C):
    import torch
    _expect(Wqkv, torch.bfloat16, (3 * C, C), "Wqkv")
    _expect(bqkv, torch.float32, (3 * C,), "bqkv")
    _expect(Wo, torch.bfloat16, (C, C), "Wo")
    _expect(bo, torch.float32, (C,), "bo")


def dfa_qkv_proj(X, Wqkv, bqkv, Q, K, V, stream=None) -> None:
    """Q, K, V = split(X Wqkv^T + bqkv); X [B, L, H*d] bf16, Q/K/V [B, H, L, d] bf16."""
    import torch
    B, H, L, d = _shape(Q, K, V)
    _proj_shapes(X, Q)
    _expect(X, torch.bfloat16, X.shape, "X")
    _weights(Wqkv, bqkv, None, None, H * d)
    _check(lib().dfa_qkv_proj(_ptr(X), _ptr(Wqkv), _ptr(bqkv), _ptr(Q), _ptr(K), _ptr(V), B, H, L, d, _stream(stream)))


def dfa_out_proj(O, Wo, bo, Y, stream=None) -> None:
    """Y = merge(O) Wo^T + bo; O [B, H, L, d] bf16, Y [B, L, H*d] bf16."""
    import torch
    B, H, L, d = _shape(O)
    _proj_shapes(Y, O)
    _expect(Y, torch.bfloat16, Y.shape, "Y")
    _weights(None, None, Wo, bo, H * d)
    _check(lib().dfa_out_proj(_ptr(O), _ptr(Wo), _ptr(bo), _ptr(Y), B, H, L, d, _stream(stream)))


def dfa_module_step(code: int, X, Wqkv, bqkv, Wo, bo, Q, K, V, O, R, Y, Ycache, w: int, H: int,
                    stream=None) -> None:
    """One attention module with H heads under a plan code (see include/dfa.h).
    Shapes come from Y [B, L, C] (d = C / H); for AST every other tensor may
    be None."""
    import torch
    if Y is None or Y.dim() != 3:
        raise ValueError("Y must be a [B, L, C] tensor")
    B, L, C = Y.shape
    if H <= 0 or C % H:
        raise ValueError(f"C={C} is not a multiple of H={H}")
    d = C // H
    for t, name in ((X, "X"), (Y, "Y"), (Ycache, "Ycache")):
        _expect(t, torch.bfloat16, (B, L, C), name)
    for t, name in ((Q, "Q"), (K, "K"), (V, "V"), (O, "O")):
        _expect(t, torch.bfloat16, (B, H, L, d), name)
    _expect(R, torch.float32, (B, H, L, d), "R")
    _weights(Wqkv, bqkv, Wo, bo, C)
    _check(lib().dfa_module_step(int(code), _ptr(X), _ptr(Wqkv), _ptr(bqkv), _ptr(Wo), _ptr(bo), _ptr(Q), _ptr(K),
                                 _ptr(V), _ptr(O), _ptr(R), _ptr(Y), _ptr(Ycache), B, H, L, d, w, _stream(stream)))


def _on_gpu(*named):
    for t, name in named:
        if t.device.type != "cuda" or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous GPU tensor (got {t.device})")


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def dfa_mrae(A, B, workspace, result, stream=None) -> None:
    """result (a 1-element fp64 GPU tensor) = MRAE of two bf16 tensors of the
    same size; workspace: a GPU tensor of at least MRAE_WORKSPACE_BYTES bytes."""
    import torch
    if A.dtype != torch.bfloat16 or B.dtype != torch.bfloat16 or A.numel() != B.numel():
        raise ValueError("A and B must be bf16 tensors of the same size")
    _on_gpu((A, "A"), (B, "B"), (workspace, "workspace"), (result, "result"))
    if _nbytes(workspace) < MRAE_WORKSPACE_BYTES or result.dtype != torch.float64 or result.numel() < 1:
        raise ValueError("workspace too small or result not an fp64 tensor")
    _check(lib().dfa_mrae(_ptr(A), _ptr(B), A.numel(), _ptr(workspace), _ptr(result), _stream(stream)))


def dfa_mrae_noalloc(A, B, result, stream=None) -> None:
    """dfa_mrae without a workspace: the library keeps the partial sums in a
    device array of its own (no allocation by the call)."""
    import torch
    if A.dtype != torch.bfloat16 or B.dtype != torch.bfloat16 or A.numel() != B.numel():
        raise ValueError("A and B must be bf16 tensors of the same size")
    _on_gpu((A, "A"), (B, "B"), (result, "result"))
    if result.dtype != torch.float64 or result.numel() < 1:
        raise ValueError("result must be an fp64 tensor")
    _check(lib().dfa_mrae_noalloc(_ptr(A), _ptr(B), A.numel(), _ptr(result), _stream(stream)))


def plan_search_workspace_bytes(n_layers: int, B: int, H: int, L: int, d: int) -> int:
    return int(lib().dfa_plan_search_workspace_bytes(n_layers, B, H, L, d))


def dfa_plan_search(X_steps, layers, delta: float, w: int, H: int, workspace, stream=None):
    """Greedy plan search (see include/dfa.h) over hidden states X_steps (list of
    [B, L, C] bf16 GPU tensors) and layers (list of (Wqkv, bqkv, Wo, bo) GPU
    tensors); workspace: a GPU tensor of at least plan_search_workspace_bytes()
    bytes.  Biases are given for every layer or for none.
    Returns (plan int32 [T, n_layers], loss float64 [T, n_layers])."""
    import torch
    if not X_steps or not layers:
        raise ValueError("X_steps and layers must be non-empty")
    B, L, C = X_steps[0].shape
    if H <= 0 or C % H:
        raise ValueError(f"C={C} is not a multiple of H={H}")
    d = C // H
    for X in X_steps:
        _expect(X, torch.bfloat16, (B, L, C), "X_steps[t]")
    for Wqkv, bqkv, Wo, bo in layers:
        _weights(Wqkv, bqkv, Wo, bo, C)
    _on_gpu((workspace, "workspace"))
    T, n = len(X_steps), len(layers)
    arr = lambda ts: (ctypes.c_void_p * len(ts))(*[_ptr(t) for t in ts])  # noqa: E731
    biased = [(l[1] is not None, l[3] is not None) for l in layers]
    has_b = all(a and b for a, b in biased)
    if not has_b and any(a or b for a, b in biased):
        raise ValueError("give both biases for every layer or for none")
    plan = np.full((T, n), -1, dtype=np.int32)
    loss = np.full((T, n), np.nan)
    _check(lib().dfa_plan_search(n, T, arr(X_steps), arr([l[0] for l in layers]),
                                 arr([l[1] for l in layers]) if has_b else None, arr([l[2] for l in layers]),
                                 arr([l[3] for l in layers]) if has_b else None, float(delta), B, H, L, d, w,
                                 _ptr(workspace), _nbytes(workspace), plan.ctypes.data_as(_i32p),
                                 loss.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), _stream(stream)))
    return plan, loss


def dfa_plan_make(seed: int, n_layers: int, n_steps: int, refresh_every: int, B: int):
    """Seeded plan: int32 arrays (code, r_src, o_src) of shape [n_steps, n_layers]."""
    shape = (max(n_steps, 0), max(n_layers, 0))
    code = np.full(shape, -1, dtype=np.int32)
    r_src = np.full(shape, -1, dtype=np.int32)
    o_src = np.full(shape, -1, dtype=np.int32)
    as_p = lambda a: a.ctypes.data_as(_i32p)  # noqa: E731
    _check(lib().dfa_plan_make(ctypes.c_uint64(seed & (2**64 - 1)), n_layers, n_steps, refresh_every, B,
                               as_p(code), as_p(r_src), as_p(o_src)))
    return code, r_src, o_src


def version() -> str:
    return lib().dfa_version().decode()
