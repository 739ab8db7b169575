"""Seeded random-shape parity sweep of the attention entry points.

Each case draws (B, H, L, d, w) from a fixed generator: L log-uniform from 1
to about 2800 tokens, half-widths from 0 through the sequence length to the
largest int.  Every entry point runs into outputs with guard bands and is
checked against the fp64 oracle to the bounds of `test_gpu_parity.check`;
even batches also run ASC and the combined WA-RS + ASC refresh and reuse
through `dfa_plan_step`.  This sweep found that rows of a few keys needed
split probabilities (three-key rows missed the 1e-2 bound)."""
import random

import numpy as np
import pytest
import torch

from oracle import dfa_oracle as orc
from paper_2406_08552_amd import dfa
from tests.test_gpu_parity import Guarded, check, f64, rand_qkv, say

N_CASES = 60


def draw_cases(seed: int, n: int):
    rng = random.Random(seed)
    cases = []
    for _ in range(n):
        d = rng.choice([64, 72])
        L = max(1, int(round(10 ** rng.uniform(0, 3.45))))
        B, H = rng.choice([1, 2, 2, 3, 4]), rng.choice([1, 2, 3, 5])
        while B * H * L * L > 40e6 and (B > 1 or H > 1):   # bounds the oracle's work
            if B > 1:
                B -= 1
            else:
                H -= 1
        w = rng.choice([0, 1, rng.randint(0, max(0, L // 4)), L // 8, max(0, L - 2), max(0, L - 1), L,
                        2 ** 31 - 1, rng.randint(0, L + 5)])
        cases.append((B, H, L, d, w))
    return cases


@pytest.mark.gpu
@pytest.mark.parametrize("case,B,H,L,d,w", [(i, *c) for i, c in enumerate(draw_cases(20261202, N_CASES))])
def test_random_shape(case, B, H, L, d, w):
    dev = torch.device("cuda")
    shape = (B, H, L, d)
    say(f"sweep case {case}: B={B} H={H} L={L} d={d} w={w}")
    q, k, v = rand_qkv(shape, 5000 + case)
    gq, gk, gv = (t.to(dev) for t in (q, k, v))
    Qd, Kd, Vd = f64(q), f64(k), f64(v)
    Of = orc.attn_full(Qd, Kd, Vd)
    Wd = orc.attn_window(Qd, Kd, Vd, w)
    Rres = (torch.randn(shape, generator=torch.Generator().manual_seed(77 + case)) * 0.1).float()
    O1, O2, O3, O4 = (Guarded(shape, dev) for _ in range(4))
    R2 = Guarded(shape, dev, torch.float32)
    dfa.dfa_attn_full(gq, gk, gv, O1.t, w)
    dfa.dfa_attn_full_and_residual(gq, gk, gv, O2.t, R2.t, w)
    dfa.dfa_attn_window_plus_residual(gq, gk, gv, O3.t, Rres.to(dev), w)
    dfa.dfa_attn_window_plus_residual(gq, gk, gv, O4.t, None, w)
    torch.cuda.synchronize()
    for name, got, ref in (("full", O1, Of), ("refresh O", O2, Of), ("refresh R", R2, Of - Wd),
                           ("window + R", O3, Wd + f64(Rres)), ("window", O4, Wd)):
        assert got.guards_intact(), f"{name}: write outside the tensor"
        check(name, got.t, ref)
    if w >= L - 1:
        assert torch.equal(R2.t, torch.zeros_like(R2.t)), "a band covering every key must give R == 0 exactly"
        assert torch.equal(O4.t, O1.t), "a band covering every key must reproduce full attention bitwise"
    if B % 2:
        return
    h = B // 2
    Oc = torch.empty(shape, dtype=torch.bfloat16, device=dev)
    R5 = torch.zeros(shape, dtype=torch.float32, device=dev)
    O5, O6, O7 = (Guarded(shape, dev) for _ in range(3))
    dfa.dfa_plan_step(dfa.ASC_REUSE, gq, gk, gv, O5.t, None, Oc, w)
    dfa.dfa_plan_step(dfa.WARS_ASC_REFRESH, gq, gk, gv, O6.t, R5, Oc, w)
    dfa.dfa_plan_step(dfa.WARS_ASC_REUSE, gq, gk, gv, O7.t, R5, Oc, w)
    torch.cuda.synchronize()
    assert O5.guards_intact() and O6.guards_intact() and O7.guards_intact()
    for O in (O5, O6, O7):
        assert torch.equal(O.t[:h], O.t[h:]), "CFG-shared halves must be bit-identical"
    check("asc", O5.t[:h], Of[:h])
    Oref, Rc = orc.wars_asc_refresh(Qd, Kd, Vd, w)
    check("wars+asc refresh O", O6.t, Oref)
    check("wars+asc refresh R", R5[:h], Rc)
    assert torch.equal(R5[h:], torch.zeros_like(R5[h:])), "a half-batch refresh must leave R[uncond]"
    check("wars+asc reuse", O7.t, orc.wars_asc_reuse(Qd, Kd, Vd, Rc, w))


def test_sweep_draws_are_fixed():
    """The drawn shapes are a function of the seed only (a CPU-side check of
    the generator the GPU cases use)."""
    a, b = draw_cases(20261202, N_CASES), draw_cases(20261202, N_CASES)
    assert a == b and len(set(a)) > N_CASES // 2
    assert any(c[2] <= 32 for c in a) and any(c[2] > 1000 for c in a)
    assert any(c[4] >= c[2] - 1 for c in a) and any(c[4] <= 1 for c in a)
    assert np.mean([c[3] == 72 for c in a]) > 0.2


N_LARGE = 24


def draw_large_cases(seed: int, n: int):
    """Launches of more than 256 128-query workgroups (the two-block kernels):
    L from 300 to 9000 tokens and B*H to match, half-widths from 0 to beyond L."""
    rng = random.Random(seed)
    cases = []
    for _ in range(n):
        d = rng.choice([64, 72])
        L = int(round(10 ** rng.uniform(np.log10(300), np.log10(9000))))
        bh_min = 257 * 128 // L + 1
        B = rng.choice([2, 4, 8])
        H = max(1, -(-bh_min // B)) + rng.randint(0, 3)
        w = rng.choice([0, 3, 16, rng.randint(17, 200), L // 8, rng.randint(0, L), max(0, L - 2), L - 1, 2 ** 31 - 1])
        cases.append((B, H, L, d, w))
    return cases


@pytest.mark.gpu
@pytest.mark.parametrize("case,B,H,L,d,w", [(i, *c) for i, c in enumerate(draw_large_cases(4242, N_LARGE))])
def test_random_large_launch(case, B, H, L, d, w):
    """Checked on 40 sampled query rows of every (batch, head): both sequence
    ends, the rows around the first query-block boundaries, and a seeded sample."""
    dev = torch.device("cuda")
    shape = (B, H, L, d)
    say(f"large sweep case {case}: B={B} H={H} L={L} d={d} w={w}")
    q, k, v = rand_qkv(shape, 7000 + case)
    Rres = rand_qkv(shape, 7100 + case)[0].float() * 0.1
    gq, gk, gv, gr = (t.to(dev) for t in (q, k, v, Rres))
    O1, O2, O3 = (torch.empty(shape, dtype=torch.bfloat16, device=dev) for _ in range(3))
    R2 = torch.empty(shape, dtype=torch.float32, device=dev)
    dfa.dfa_attn_full(gq, gk, gv, O1, w)
    dfa.dfa_attn_full_and_residual(gq, gk, gv, O2, R2, w)
    dfa.dfa_attn_window_plus_residual(gq, gk, gv, O3, gr, w)
    torch.cuda.synchronize()
    fixed = [0, 1, 63, 64, 127, 128, 129, L // 2, L - 129, L - 128, L - 65, L - 64, L - 2, L - 1]
    rows = np.unique(np.concatenate([fixed, np.random.default_rng(7200 + case).integers(0, L, 26)]))
    Qd, Kd, Vd = f64(q), f64(k), f64(v)
    Of = orc.attention_rows(Qd, Kd, Vd, rows, None)
    Wd = orc.attention_rows(Qd, Kd, Vd, rows, w)
    check("full", O1, Of, rows)
    check("refresh O", O2, Of, rows)
    check("refresh R", R2, Of - Wd, rows)
    check("window + R", O3, Wd + f64(Rres)[:, :, rows], rows)


def test_large_draws_take_two_block_kernels():
    """Every large case launches more than 256 128-query workgroups."""
    for B, H, L, d, w in draw_large_cases(4242, N_LARGE):
        assert B * H * -(-L // 128) > 256 and 300 <= L <= 9000
