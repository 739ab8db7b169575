"""The C-ABI library on the host (no GPU): it loads, exports every symbol the
header declares, rejects bad arguments before touching a device, and its plan
generator equals the oracle's bit for bit."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import dfa_oracle as orc
from paper_2406_08552_amd import dfa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dfa.h")


@pytest.fixture(scope="module")
def L():
    return dfa.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dfa_[a-z_]+)\s*\(", text)))


def test_header_declares_binding_exports():
    assert declared_functions() == sorted(dfa.EXPORTS)


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), name
    assert dfa.version().count(".") == 2


# Addresses that are never dereferenced: validation fails before any HIP call.
A, B_, C_, D_, E_ = (0x10000 * (i + 1) for i in range(5))


def call_full(L, Q=A, K=B_, V=C_, O=D_, B=2, H=2, L_=64, d=72, w=8):
    return L.dfa_attn_full(Q, K, V, O, None, B, H, L_, d, w, None)


@pytest.mark.parametrize("kw,status", [
    (dict(Q=None), dfa.DFA_ERR_INVALID_ARG),
    (dict(K=None), dfa.DFA_ERR_INVALID_ARG),
    (dict(O=None), dfa.DFA_ERR_INVALID_ARG),
    (dict(Q=A + 8), dfa.DFA_ERR_INVALID_ARG),          # misaligned
    (dict(B=0), dfa.DFA_ERR_INVALID_ARG),
    (dict(H=-1), dfa.DFA_ERR_INVALID_ARG),
    (dict(L_=0), dfa.DFA_ERR_INVALID_ARG),
    (dict(d=0), dfa.DFA_ERR_INVALID_ARG),
    (dict(w=-1), dfa.DFA_ERR_INVALID_ARG),
    (dict(d=80), dfa.DFA_ERR_UNSUPPORTED),
    (dict(d=60), dfa.DFA_ERR_UNSUPPORTED),
    (dict(O=A), dfa.DFA_ERR_INVALID_ARG),              # O aliases Q
    (dict(O=B_ + 64), dfa.DFA_ERR_INVALID_ARG),        # O overlaps K
])
def test_full_validation(L, kw, status):
    assert call_full(L, **kw) == status
    assert dfa.last_error()


def test_refresh_validation(L):
    f = L.dfa_attn_full_and_residual
    assert f(A, B_, C_, D_, None, 2, 2, 64, 72, 8, None) == dfa.DFA_ERR_INVALID_ARG   # R missing
    assert f(A, B_, C_, D_, D_, 2, 2, 64, 72, 8, None) == dfa.DFA_ERR_INVALID_ARG     # O == R
    assert f(A, B_, C_, D_, A, 2, 2, 64, 72, 8, None) == dfa.DFA_ERR_INVALID_ARG      # R aliases Q


def test_window_validation(L):
    f = L.dfa_attn_window_plus_residual
    assert f(A, B_, C_, D_, D_, 2, 2, 64, 72, 8, None) == dfa.DFA_ERR_INVALID_ARG     # O == R
    assert f(A, B_, C_, D_, E_ + 4, 2, 2, 64, 72, 8, None) == dfa.DFA_ERR_INVALID_ARG  # misaligned R
    assert f(A, B_, C_, D_, None, 2, 2, 64, 72, -3, None) == dfa.DFA_ERR_INVALID_ARG


def test_plan_step_validation(L):
    f = L.dfa_plan_step
    args = (2, 2, 64, 72, 8, None)
    assert f(7, A, B_, C_, D_, E_, None, *args) == dfa.DFA_ERR_INVALID_ARG            # unknown code
    assert f(-1, A, B_, C_, D_, E_, None, *args) == dfa.DFA_ERR_INVALID_ARG
    assert f(dfa.WARS_REFRESH, A, B_, C_, D_, None, None, *args) == dfa.DFA_ERR_INVALID_ARG
    assert f(dfa.WARS_REUSE, A, B_, C_, D_, None, None, *args) == dfa.DFA_ERR_INVALID_ARG
    assert f(dfa.AST_REUSE, None, None, None, D_, None, None, *args) == dfa.DFA_ERR_INVALID_ARG
    assert "Ocache" in dfa.last_error()
    # AST with the cache equal to O is a no-op: OK without any device work
    assert f(dfa.AST_REUSE, None, None, None, D_, None, D_, *args) == dfa.DFA_OK
    for code in (dfa.ASC_REUSE, dfa.WARS_ASC_REFRESH, dfa.WARS_ASC_REUSE):
        assert f(code, A, B_, C_, D_, E_, None, 3, 2, 64, 72, 8, None) == dfa.DFA_ERR_INVALID_ARG
        assert "even" in dfa.last_error()
    for code in (dfa.WARS_ASC_REFRESH, dfa.WARS_ASC_REUSE):
        assert f(code, A, B_, C_, D_, None, None, *args) == dfa.DFA_ERR_INVALID_ARG   # R missing
        assert "R is NULL" in dfa.last_error()
        assert f(code, A, B_, C_, D_, D_, None, *args) == dfa.DFA_ERR_INVALID_ARG     # O == R
    assert f(dfa.FULL, A, B_, C_, D_, None, D_ + 32, *args) == dfa.DFA_ERR_INVALID_ARG  # cache overlaps O
    assert f(dfa.FULL, A, B_, C_, D_, None, A, *args) == dfa.DFA_ERR_INVALID_ARG       # cache aliases Q
    assert f(dfa.FULL, None, B_, C_, D_, None, None, *args) == dfa.DFA_ERR_INVALID_ARG


def test_error_message_is_per_call(L):
    call_full(L, d=80)
    assert "d=80" in dfa.last_error()
    call_full(L, w=-5)
    assert "w=-5" in dfa.last_error()


PLAN_CASES = [(28, 50, 0, 8), (28, 20, 4, 2), (3, 40, 2, 2), (5, 30, 0, 4), (1, 1, 0, 2), (2, 7, 1, 2),
              (4, 9, 3, 6)]


@pytest.mark.parametrize("n_layers,n_steps,every,B", PLAN_CASES)
def test_plan_bit_equal_to_oracle(n_layers, n_steps, every, B):
    for seed in list(range(0, 1000, 7)) + [240608552 + 2, 240608552 + 5, 2**64 - 1, 2**63]:
        ours = dfa.dfa_plan_make(seed, n_layers, n_steps, every, B)
        ref = orc.plan_make(seed, n_layers, n_steps, every, B)
        for a, b in zip(ours, ref):
            assert a.dtype == np.int32 and np.array_equal(a, b), (seed, n_layers, n_steps, every, B)


def test_plan_odd_batch_and_bad_dims():
    with pytest.raises(dfa.DfaError) as e:
        # 28 x 50 draws contain ASC for this seed
        dfa.dfa_plan_make(5, 28, 50, 0, 3)
    assert e.value.status == dfa.DFA_ERR_INVALID_ARG
    with pytest.raises(ValueError):
        orc.plan_make(5, 28, 50, 0, 3)
    for bad in ((0, 5, 0, 2), (5, 0, 0, 2), (5, 5, -1, 2), (5, 5, 0, 0)):
        with pytest.raises(dfa.DfaError):
            dfa.dfa_plan_make(1, *bad)


def test_plan_null_arrays(L):
    assert L.dfa_plan_make(ctypes.c_uint64(1), 2, 2, 0, 2, None, None, None) == dfa.DFA_ERR_INVALID_ARG


def test_size_limits(L):
    """Token counts that the kernels' int index arithmetic cannot hold are
    rejected before any launch (the tensors themselves would fit in HBM)."""
    f = L.dfa_attn_full
    assert f(A, B_, C_, D_, None, 1, 1, (1 << 30) + 1, 64, 8, None) == dfa.DFA_ERR_INVALID_ARG
    assert "too large" in dfa.last_error()
    big = 0x1000000
    X, W, Q, K, V = (big * (i + 1) for i in range(5))
    # B * L = 2^31 tokens at C = 128: 2^38 elements, within the tensor limit
    assert L.dfa_qkv_proj(X, W, None, Q, K, V, 2, 2, 1 << 30, 64, None) == dfa.DFA_ERR_INVALID_ARG
    assert "B*L" in dfa.last_error()
    assert L.dfa_out_proj(Q, W, None, X, 2, 2, 1 << 30, 64, None) == dfa.DFA_ERR_INVALID_ARG


def test_projection_validation(L):
    fq, fo, fm = L.dfa_qkv_proj, L.dfa_out_proj, L.dfa_module_step
    big = 0x1000000
    X, W, Q, K, V = (big * (i + 1) for i in range(5))
    assert fq(X, W, None, Q, K, V, 2, 3, 64, 72, None) == dfa.DFA_ERR_UNSUPPORTED   # C = 216
    assert "multiple of 128" in dfa.last_error()
    assert fq(X, W, None, Q, K, V, 2, 16, 64, 80, None) == dfa.DFA_ERR_UNSUPPORTED
    assert fq(None, W, None, Q, K, V, 2, 16, 64, 72, None) == dfa.DFA_ERR_INVALID_ARG
    assert fq(X, W, X + 4, Q, K, V, 2, 16, 64, 72, None) == dfa.DFA_ERR_INVALID_ARG   # misaligned bias
    assert fq(X, W, None, X, K, V, 2, 16, 64, 72, None) == dfa.DFA_ERR_INVALID_ARG    # Q aliases X
    assert fq(X, W, None, Q, Q + 64, V, 2, 16, 64, 72, None) == dfa.DFA_ERR_INVALID_ARG  # K overlaps Q
    assert fo(Q, W, None, Q, 2, 16, 64, 72, None) == dfa.DFA_ERR_INVALID_ARG           # Y aliases O
    assert fo(Q, W, None, None, 2, 16, 64, 72, None) == dfa.DFA_ERR_INVALID_ARG
    args = (2, 16, 64, 72, 8, None)
    R, O, Y, Yc, Wo = (big * (i + 10) for i in range(5))
    assert fm(9, X, W, None, Wo, None, Q, K, V, O, R, Y, Yc, *args) == dfa.DFA_ERR_INVALID_ARG   # code
    assert fm(dfa.AST_REUSE, None, None, None, None, None, None, None, None, None, None, Y, None, *args) \
        == dfa.DFA_ERR_INVALID_ARG
    assert "Ycache" in dfa.last_error()
    assert fm(dfa.AST_REUSE, None, None, None, None, None, None, None, None, None, None, Y, Y, *args) == dfa.DFA_OK
    assert fm(dfa.ASC_REUSE, X, W, None, Wo, None, Q, K, V, O, R, Y, Yc, 3, 16, 64, 72, 8, None) \
        == dfa.DFA_ERR_INVALID_ARG
    assert "even" in dfa.last_error()
    assert fm(dfa.WARS_REFRESH, X, W, None, Wo, None, Q, K, V, O, None, Y, Yc, *args) == dfa.DFA_ERR_INVALID_ARG
    assert "R is NULL" in dfa.last_error()
    assert fm(dfa.FULL, X, W, None, Wo, None, Q, K, V, Q, R, Y, Yc, *args) == dfa.DFA_ERR_INVALID_ARG  # O == Q
    assert fm(dfa.FULL, X, W, None, Wo, None, Q, K, V, O, R, Y, Y + 64, *args) == dfa.DFA_ERR_INVALID_ARG
    assert fm(dfa.FULL, X, W, None, Wo, None, Q, K, V, O, R, X, Yc, *args) == dfa.DFA_ERR_INVALID_ARG  # Y == X
    assert fm(dfa.FULL, X, W, None, Wo, None, Q, K, V, O, R, Y, Yc, 2, 16, 64, 72, -1, None) == dfa.DFA_ERR_INVALID_ARG


def test_search_and_mrae_validation(L):
    import ctypes
    assert L.dfa_mrae(None, 0x1000, 8, 0x2000, 0x3000, None) == dfa.DFA_ERR_INVALID_ARG
    assert L.dfa_mrae(0x1008, 0x1000, 8, 0x2000, 0x3000, None) == dfa.DFA_ERR_INVALID_ARG   # misaligned
    assert "aligned" in dfa.last_error()
    assert L.dfa_mrae_noalloc(None, 0x1000, 8, 0x3000, None) == dfa.DFA_ERR_INVALID_ARG
    assert L.dfa_mrae_noalloc(0x1000, 0x1000, 8, 0x3004, None) == dfa.DFA_ERR_INVALID_ARG   # misaligned result
    assert L.dfa_mrae_noalloc(0x1000, 0x1000, (1 << 40) + 1, 0x3000, None) == dfa.DFA_ERR_INVALID_ARG
    assert "2^40" in dfa.last_error()
    assert dfa.plan_search_workspace_bytes(3, 2, 2, 64, 64) > 0
    assert dfa.plan_search_workspace_bytes(0, 2, 2, 64, 64) == 0
    f = L.dfa_plan_search
    ptrs = (ctypes.c_void_p * 2)(0x100000, 0x200000)
    plan = np.zeros(4, dtype=np.int32)
    loss = np.zeros(4)
    pp = plan.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    lp = loss.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    need = dfa.plan_search_workspace_bytes(2, 2, 2, 64, 64)
    args = (2, 2, ptrs, ptrs, None, ptrs, None)
    assert f(*args, -1.0, 2, 2, 64, 64, 8, 0x400000, need, pp, lp, None) == dfa.DFA_ERR_INVALID_ARG   # delta < 0
    assert f(*args, 0.1, 2, 3, 64, 64, 8, 0x400000, need, pp, lp, None) == dfa.DFA_ERR_UNSUPPORTED    # C = 192
    assert f(*args, 0.1, 2, 2, 64, 64, 8, 0x400000, need - 1, pp, lp, None) == dfa.DFA_ERR_INVALID_ARG
    assert "too small" in dfa.last_error()
    assert f(*args, 0.1, 2, 2, 64, 64, 8, 0x400010, need, pp, lp, None) == dfa.DFA_ERR_INVALID_ARG
    assert f(*args, 0.1, 2, 2, 64, 64, 8, 0x400000, need, None, lp, None) == dfa.DFA_ERR_INVALID_ARG


def test_binding_rejects_host_tensors():
    """The binding refuses host tensors before any device pointer reaches the
    library (a host address written by a kernel would fault the GPU)."""
    import torch
    a = torch.zeros(64, dtype=torch.bfloat16)
    ws = torch.zeros(dfa.MRAE_WORKSPACE_BYTES, dtype=torch.uint8)
    res = torch.zeros(1, dtype=torch.float64)
    with pytest.raises(ValueError, match="GPU"):
        dfa.dfa_mrae(a, a, ws, res)
    with pytest.raises(ValueError, match="non-empty"):
        dfa.dfa_plan_search([], [], 0.1, 4, 2, ws)
    q = torch.zeros((1, 1, 64, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU"):
        dfa.dfa_attn_full(q, q, q, q.clone(), 0)


def test_binding_fails_loudly_without_the_library(tmp_path):
    """With no built library the binding raises on first use; there is no
    fallback path (checked in a fresh interpreter pointed at a missing file)."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("from paper_2406_08552_amd import dfa\n"
            "try:\n    dfa.lib()\nexcept RuntimeError as e:\n    print('raised:', e)\n")
    env = dict(os.environ, DFA_LIBRARY=str(tmp_path / "libdfa_missing.so"))
    out = subprocess.run([sys.executable, "-c", code], cwd=root, env=env, capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    assert "raised:" in out.stdout and "is missing" in out.stdout, out.stdout
