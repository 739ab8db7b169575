"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Floating-point outputs must satisfy max|gpu - oracle| <= 1e-2 and
mean|gpu - oracle| <= 1e-3 (unit-variance inputs); plan arrays, AST copies
and ASC halves must match bit for bit.  A bf16 output cannot be closer to
the exact value than its correct rounding: where that floor itself exceeds a
bound (outputs of unit magnitude, e.g. a band of half-width 0 whose window
output is V, reach 4 and more, where half a bf16 ulp is 0.0156), the bound is
1.1 x (mean) or 1.25 x (max) the error of the oracle's own result rounded to
bf16.  Long sequences are checked on a
seeded sample of query rows (rows are independent, so the sampled oracle
carries its own per-row caches).
"""
import numpy as np
import pytest
import torch

from oracle import dfa_oracle as orc
from paper_2406_08552_amd import dfa, inputs

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS = 1e-2, 1e-3
f64 = inputs.as_f64


def say(msg):
    print(f"[gpu] {msg}", flush=True)


def rand_qkv(shape, seed):
    g = torch.Generator().manual_seed(seed)
    return tuple(torch.randn(shape, generator=g).to(torch.bfloat16) for _ in range(3))


def bf16_floor(ref):
    """Mean and max error of the exact result correctly rounded to bf16."""
    r = torch.from_numpy(np.ascontiguousarray(ref)).to(torch.bfloat16).to(torch.float64).numpy()
    e = np.abs(r - ref)
    return float(e.mean()), float(e.max())


def check(name, got, ref, rows=None, max_abs=MAX_ABS):
    g = f64(got)
    if rows is not None:
        g = g[:, :, rows]
    err = np.abs(g - ref)
    assert np.all(np.isfinite(g)), f"{name}: non-finite output"
    mx, mn = float(err.max()), float(err.mean())
    mean_bar, max_bar = MEAN_ABS, max_abs
    if got.dtype == torch.bfloat16:
        fmean, fmax = bf16_floor(ref)
        mean_bar, max_bar = max(MEAN_ABS, 1.1 * fmean), max(max_abs, 1.25 * fmax)
    assert mx <= max_bar and mn <= mean_bar, \
        f"{name}: max abs {mx:.3e} (bar {max_bar:.3e}), mean abs {mn:.3e} (bar {mean_bar:.3e})"
    return mx, mn


class Guarded:
    """A [B,H,L,d] device tensor with sentinel guard bands on both sides: any
    write outside the tensor shows up in the guards."""
    PAD = 4096

    def __init__(self, shape, dev, dtype=torch.bfloat16):
        n = int(np.prod(shape))
        self.dtype = dtype
        self.buf = torch.full((n + 2 * self.PAD,), 12345.0, dtype=dtype, device=dev)
        self.t = self.buf[self.PAD:self.PAD + n].view(shape)

    def guards_intact(self):
        sentinel = torch.tensor(12345.0, dtype=self.dtype)
        lo, hi = self.buf[:self.PAD].cpu(), self.buf[-self.PAD:].cpu()
        return bool(torch.all(lo == sentinel)) and bool(torch.all(hi == sentinel))


SHAPES = [  # (B, H, L, d, w): tiles, ragged tails, degenerate bands
    (1, 1, 64, 64, 0),
    (2, 2, 256, 64, 16),
    (1, 2, 200, 72, 24),
    (1, 1, 77, 72, 5),
    (2, 1, 130, 72, 129),
    (1, 1, 1, 72, 0),
    (1, 1, 17, 64, 3),
    (1, 2, 1000, 72, 125),
    (2, 2, 300, 72, 0),
    (1, 1, 129, 64, 1000),
    (1, 1, 513, 72, 1),
    (3, 1, 384, 72, 64),
    # short sequences (one wavefront per sequence): B*H not a multiple of the
    # four sequences of a workgroup, one and two 16-key blocks, bands covering
    # every key, and the first length that takes the tiled kernels again
    (3, 5, 16, 72, 2),
    (2, 3, 32, 72, 31),
    (1, 2, 31, 72, 4),
    (2, 2, 12, 64, 0),
    (1, 3, 25, 64, 30),
    (1, 1, 33, 72, 3),
]


@pytest.mark.parametrize("B,H,L,d,w", SHAPES)
def test_kernels_vs_oracle(B, H, L, d, w):
    dev = torch.device("cuda")
    shape = (B, H, L, d)
    q, k, v = rand_qkv(shape, 1000 + L + w + d)
    Rres = rand_qkv(shape, 7 + L)[0].float() * 0.1
    gq, gk, gv, gr = (t.to(dev) for t in (q, k, v, Rres))
    O1, O2, O3 = (Guarded(shape, dev) for _ in range(3))
    R2 = Guarded(shape, dev, torch.float32)
    say(f"kernels B={B} H={H} L={L} d={d} w={w}")
    dfa.dfa_attn_full(gq, gk, gv, O1.t, w)
    dfa.dfa_attn_full_and_residual(gq, gk, gv, O2.t, R2.t, w)
    dfa.dfa_attn_window_plus_residual(gq, gk, gv, O3.t, gr, w)
    torch.cuda.synchronize()
    Qd, Kd, Vd = f64(q), f64(k), f64(v)
    Of = orc.attn_full(Qd, Kd, Vd)
    Wd = orc.attn_window(Qd, Kd, Vd, w)
    check("full", O1.t, Of)
    check("refresh O", O2.t, Of)
    check("refresh R", R2.t, Of - Wd)
    check("window + R", O3.t, Wd + f64(Rres))
    for gbuf in (O1, O2, R2, O3):
        assert gbuf.guards_intact(), "write outside the output tensor"
    # the refresh output is full attention from the same kernel family
    if w >= L - 1:
        assert not torch.any(R2.t.cpu().float() != 0), "w >= L-1 must give R == 0 exactly"
        O4 = torch.empty(shape, dtype=torch.bfloat16, device=dev)
        dfa.dfa_attn_window_plus_residual(gq, gk, gv, O4, None, w)
        torch.cuda.synchronize()
        assert torch.equal(O4, O1.t), "a band covering every key must reproduce full attention bitwise"


# Launches with short tile walks, or with at most 256 workgroups of 128
# queries, run 64-query workgroups (one 16-query block per wavefront), the
# rest 128-query workgroups; these shapes sit on both sides of each switch:
# full attention at L = 256, refresh at L = 512 (one pass with two
# accumulators up to there) and at L = 1024, window attention at a band of
# 1280 keys (w = 639 / 640), and the workgroup count (B*H*ceil(L/128) = 256
# against 288 and 384).
ROUTE_SHAPES = [
    (1, 16, 2048, 72, 256),
    (2, 16, 1025, 72, 100),
    (2, 16, 1500, 64, 640),
    (1, 2, 256, 72, 32),
    (1, 2, 512, 64, 40),
    (2, 1, 513, 72, 40),
    (1, 2, 257, 64, 32),
    (2, 1, 1024, 72, 100),
    (1, 2, 1025, 72, 100),
    (1, 1, 1500, 64, 639),
    (1, 1, 1500, 72, 640),
    (1, 1, 2100, 72, 700),
    (1, 1, 700, 72, 699),
]


@pytest.mark.parametrize("B,H,L,d,w", ROUTE_SHAPES)
def test_query_block_routes(B, H, L, d, w):
    test_kernels_vs_oracle(B, H, L, d, w)


def test_long_sequence_sampled():
    """L = 65536 (four times the 2K workload's tokens) through the three
    kernels, on sampled query rows: the first and last rows, the rows at the
    band edges next to the sequence ends and at key-tile boundaries, and a
    seeded sample."""
    dev = torch.device("cuda")
    B, H, L, d, w = 1, 2, 65536, 72, 8192
    shape = (B, H, L, d)
    q, k, v = rand_qkv(shape, 65536)
    Rres = rand_qkv(shape, 65537)[0].float() * 0.1
    gq, gk, gv, gr = (t.to(dev) for t in (q, k, v, Rres))
    O1, O2, O3 = (torch.empty(shape, dtype=torch.bfloat16, device=dev) for _ in range(3))
    R2 = torch.empty(shape, dtype=torch.float32, device=dev)
    say(f"long sequence B={B} H={H} L={L} d={d} w={w}")
    dfa.dfa_attn_full(gq, gk, gv, O1, w)
    dfa.dfa_attn_full_and_residual(gq, gk, gv, O2, R2, w)
    dfa.dfa_attn_window_plus_residual(gq, gk, gv, O3, gr, w)
    torch.cuda.synchronize()
    fixed = [0, 1, 63, 64, 127, 128, w - 1, w, w + 1, L // 2, L - w - 2, L - w - 1, L - 129, L - 128,
             L - 65, L - 64, L - 2, L - 1]
    rows = np.unique(np.concatenate([fixed, np.random.default_rng(65536).integers(0, L, 48)]))
    Qd, Kd, Vd = f64(q), f64(k), f64(v)
    Of = orc.attention_rows(Qd, Kd, Vd, rows, None)
    Wd = orc.attention_rows(Qd, Kd, Vd, rows, w)
    check("long full", O1, Of, rows)
    check("long refresh O", O2, Of, rows)
    check("long refresh R", R2, Of - Wd, rows)
    check("long window + R", O3, Wd + f64(Rres)[:, :, rows], rows)


def test_concurrent_streams_match_serial():
    """Calls on two streams (default priority) with disjoint outputs run
    concurrently and give the same bits as the same calls made one after the
    other: the library keeps no state between calls."""
    dev = torch.device("cuda")
    shape_a, shape_b = (2, 4, 1024, 72), (1, 8, 777, 64)
    qa, ka, va = (t.to(dev) for t in rand_qkv(shape_a, 91))
    qb, kb, vb = (t.to(dev) for t in rand_qkv(shape_b, 92))
    say("two streams: refresh + reuse on one, full + short-sequence + one-pass refresh on the other")
    qs, ks, vs = (t.to(dev) for t in rand_qkv((8, 16, 16, 72), 93))
    shape_c = (1, 4, 400, 72)
    qc, kc, vc = (t.to(dev) for t in rand_qkv(shape_c, 94))

    def work(outs):
        Oa, Ra, Oa2, Ob, Os, Oc, Rc = outs
        return [lambda: dfa.dfa_attn_full_and_residual(qa, ka, va, Oa, Ra, 128),
                lambda: dfa.dfa_attn_window_plus_residual(qa, ka, va, Oa2, Ra, 128),
                lambda: dfa.dfa_attn_full(qb, kb, vb, Ob, 0),
                lambda: dfa.dfa_plan_step(dfa.WARS_REFRESH, qs, ks, vs, Os, torch.empty(qs.shape, dtype=torch.float32,
                                                                                        device=dev), None, 2),
                lambda: dfa.dfa_attn_full_and_residual(qc, kc, vc, Oc, Rc, 40)]

    def fresh():
        return (torch.empty(shape_a, dtype=torch.bfloat16, device=dev), torch.empty(shape_a, dtype=torch.float32, device=dev),
                torch.empty(shape_a, dtype=torch.bfloat16, device=dev), torch.empty(shape_b, dtype=torch.bfloat16, device=dev),
                torch.empty(qs.shape, dtype=torch.bfloat16, device=dev),
                torch.empty(shape_c, dtype=torch.bfloat16, device=dev), torch.empty(shape_c, dtype=torch.float32, device=dev))

    serial = fresh()
    for f in work(serial):
        f()
    torch.cuda.synchronize()
    conc = fresh()
    fa, fb = work(conc)[:2], work(conc)[2:]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    for _ in range(3):
        with torch.cuda.stream(s1):
            for f in fa:
                f()
        with torch.cuda.stream(s2):
            for f in fb:
                f()
    torch.cuda.synchronize()
    for a, b in zip(serial, conc):
        assert torch.equal(a, b), "concurrent streams changed a result"


def test_plan_graph_replay():
    """A plan pass captured in a HIP graph (every plan code, a separate output
    cache so that AST launches its copy, tiled and short-sequence layers)
    replays to the same bits as the same pass run eagerly, on every replay:
    the state is reset and other eager work runs between replays."""
    dev = torch.device("cuda")
    # one query block per wavefront (d = 64, one-pass refresh), two blocks (the fast update), short sequences
    layers = [((2, 2, 300, 64), 40, [dfa.WARS_REFRESH, dfa.WARS_REUSE, dfa.AST_REUSE, dfa.ASC_REUSE,
                                      dfa.WARS_ASC_REFRESH, dfa.WARS_ASC_REUSE, dfa.FULL, dfa.WARS_REUSE]),
              ((4, 16, 1100, 72), 700, [dfa.FULL, dfa.WARS_REFRESH, dfa.AST_REUSE, dfa.WARS_REUSE,
                                        dfa.WARS_ASC_REFRESH, dfa.ASC_REUSE, dfa.WARS_ASC_REUSE, dfa.WARS_REUSE]),
              ((4, 2, 24, 72), 3, [dfa.WARS_REFRESH, dfa.ASC_REUSE, dfa.WARS_REUSE, dfa.AST_REUSE,
                                   dfa.WARS_ASC_REFRESH, dfa.WARS_ASC_REUSE, dfa.FULL, dfa.AST_REUSE])]
    qkv = [tuple(t.to(dev) for t in rand_qkv(shape, 500 + i)) for i, (shape, _, _) in enumerate(layers)]
    state = [(torch.zeros(shape, dtype=torch.bfloat16, device=dev), torch.zeros(shape, dtype=torch.float32, device=dev),
              torch.zeros(shape, dtype=torch.bfloat16, device=dev)) for shape, _, _ in layers]
    snapshot = [tuple(t.clone() for t in st) for st in state]

    def plan_pass():
        for t in range(8):
            for (shape, w, codes), (q, k, v), (O, R, C) in zip(layers, qkv, state):
                dfa.dfa_plan_step(codes[t], q, k, v, O, R, C, w)

    def reset():
        for st, sn in zip(state, snapshot):
            for a, b in zip(st, sn):
                a.copy_(b)

    say("graph replay: eager reference")
    reset()
    plan_pass()
    torch.cuda.synchronize()
    ref = [tuple(t.clone() for t in st) for st in state]
    reset()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        plan_pass()
    other = torch.empty(layers[0][0], dtype=torch.bfloat16, device=dev)
    for i in range(3):
        say(f"graph replay {i}")
        reset()
        q, k, v = qkv[0]
        dfa.dfa_attn_full(q, k, v, other, 0)          # the program's own eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for li, (st, rf) in enumerate(zip(state, ref)):
            for name, a, b in zip("ORC", st, rf):
                assert torch.equal(a, b), f"replay {i}: layer {li} {name} differs from the eager pass"


@pytest.mark.parametrize("kind,L,d,w", [("large", 2048, 72, 300), ("growing", 2048, 72, 300),
                                         ("growing", 1000, 64, 77), ("large", 777, 64, 0),
                                         ("growing", 500, 72, 40), ("large", 300, 64, 0),
                                         ("growing", 200, 72, 199)])
def test_rescale_paths(kind, L, d, w):
    """Inputs that drive the online softmax's rescale: scores of large spread
    (Q and K scaled by 6, nearly one-hot rows), or scores that grow along the
    keys so that most tiles raise the running maximum by more than the rescale
    margin."""
    dev = torch.device("cuda")
    B, H = 1, 2
    shape = (B, H, L, d)
    g = torch.Generator().manual_seed(4242 + L + d)
    q, k, v = (torch.randn(shape, generator=g) for _ in range(3))
    if kind == "large":
        q, k = 6 * q, 6 * k
    else:
        u = torch.randn(d, generator=g).sign()
        ramp = torch.linspace(0, 20, L).view(1, 1, L, 1)
        q = q + 2 * u
        k = k + ramp * u
    q, k, v = (t.to(torch.bfloat16) for t in (q, k, v))
    Rres = rand_qkv(shape, 7 + L)[0].float() * 0.1
    gq, gk, gv, gr = (t.to(dev) for t in (q, k, v, Rres))
    O1, O2, O3 = (torch.empty(shape, dtype=torch.bfloat16, device=dev) for _ in range(3))
    R2 = torch.empty(shape, dtype=torch.float32, device=dev)
    say(f"rescale paths {kind} L={L} d={d} w={w}")
    dfa.dfa_attn_full(gq, gk, gv, O1, w)
    dfa.dfa_attn_full_and_residual(gq, gk, gv, O2, R2, w)
    dfa.dfa_attn_window_plus_residual(gq, gk, gv, O3, gr, w)
    torch.cuda.synchronize()
    Qd, Kd, Vd = f64(q), f64(k), f64(v)
    Of = orc.attn_full(Qd, Kd, Vd)
    Wd = orc.attn_window(Qd, Kd, Vd, w)
    check(f"{kind} full", O1, Of)
    check(f"{kind} refresh O", O2, Of)
    check(f"{kind} refresh R", R2, Of - Wd)
    check(f"{kind} window + R", O3, Wd + f64(Rres))


# A bf16 pair whose score a * b lies just under the exact rescale threshold
# 8 / c (c = log2(e) / sqrt(72) in fp32), while its probability against a
# running max of 0, 2^(a b c - 7) (shifted by 2^-7 as the kernels form it),
# rounds to 2.0 in bf16: the fast margin test of a plain tile then falls back
# to the exact form, which finds no rescale and applies the tile with the
# running max unchanged.
MARGIN_A, MARGIN_B = 1.7421875, 27.0


def test_rescale_margin_boundary():
    """Plain tiles whose largest probability lands exactly on the margin bit
    without exceeding the rescale threshold, in full attention and in the
    plain segments of the refresh and window kernels (two query blocks per
    wavefront, where the fast margin test runs)."""
    c = np.float32(1.4426950408889634 / np.sqrt(72.0))
    s = np.float32(MARGIN_A * MARGIN_B)
    assert float(s) == MARGIN_A * MARGIN_B
    thr = np.float32(np.float32(8.0) / c)
    x = np.float32(np.float64(s) * np.float64(c) - 7.0)      # fma(s, c, -7), one rounding
    p = float(np.float32(2.0 ** np.float64(x)))
    assert s < thr and p < 2.0
    assert float(torch.tensor(p).to(torch.bfloat16)) == 2.0
    dev = torch.device("cuda")
    B, H, L, d = 4, 16, 1152, 72                 # two query blocks per wavefront in all three kernels
    shape = (B, H, L, d)
    q = torch.zeros(shape)
    q[..., 0] = MARGIN_A
    k = torch.zeros(shape)
    for h in range(H):
        for t in range(1, L // 64, 2):           # odd tiles only: walks from an even tile start at max 0
            k[:, h, 64 * t + (7 * t + 3 * h) % 64, 0] = MARGIN_B
    v = torch.randn(shape, generator=torch.Generator().manual_seed(77)).to(torch.bfloat16)
    q, k = q.to(torch.bfloat16), k.to(torch.bfloat16)
    rows = inputs.sample_rows(L, 64, 99)
    Qd, Kd, Vd = f64(q), f64(k), f64(v)
    gq, gk, gv = (t.to(dev) for t in (q, k, v))
    O = torch.empty(shape, dtype=torch.bfloat16, device=dev)
    R = torch.empty(shape, dtype=torch.float32, device=dev)
    say("margin boundary: full")
    dfa.dfa_attn_full(gq, gk, gv, O, 100)
    torch.cuda.synchronize()
    Of = orc.attention_rows(Qd, Kd, Vd, rows)
    check("margin full", O.cpu(), Of, rows)
    say("margin boundary: refresh w=100")
    dfa.dfa_attn_full_and_residual(gq, gk, gv, O, R, 100)
    torch.cuda.synchronize()
    check("margin refresh O", O.cpu(), Of, rows)
    check("margin refresh R", R.cpu(), Of - orc.attention_rows(Qd, Kd, Vd, rows, 100), rows)
    say("margin boundary: window w=700")
    dfa.dfa_attn_window_plus_residual(gq, gk, gv, O, None, 700)
    torch.cuda.synchronize()
    check("margin window", O.cpu(), orc.attention_rows(Qd, Kd, Vd, rows, 700), rows)


@pytest.mark.parametrize("B,H,L,d,w", [
    (3, 2, 1236, 64, 1),    # three keys per query: the bf16 rounding of the weights alone passed the bound
    (2, 4, 1500, 72, 2),
    (2, 3, 700, 72, 15),    # widest band applied with split probabilities
    (2, 3, 700, 72, 16),    # narrowest band applied with plain bf16 probabilities
    (2, 3, 300, 64, 7),     # a narrow band at a length the one-pass refresh would take
    (1, 2, 405, 72, 5),
    (64, 16, 16, 72, 2),    # short sequences (Open-Sora temporal shape), five keys per query
    (32, 8, 7, 64, 1),
    (40, 8, 30, 72, 3),
])
def test_narrow_windows(B, H, L, d, w):
    """Windows of a few keys per query over many outputs.  With so few keys
    the bf16 rounding of each probability (up to 2^-8 relative) does not
    average out; together with the bf16 rounding of the output it took the
    max error past 1e-2 on three-key rows.  Such rows are applied with each
    probability split into a bf16 value and its bf16 rounding residual."""
    dev = torch.device("cuda")
    shape = (B, H, L, d)
    q, k, v = rand_qkv(shape, 6100 + L + w + d)
    gq, gk, gv = (t.to(dev) for t in (q, k, v))
    Qd, Kd, Vd = f64(q), f64(k), f64(v)
    Of = orc.attn_full(Qd, Kd, Vd)
    Wd = orc.attn_window(Qd, Kd, Vd, w)
    Rres = rand_qkv(shape, 17 + L)[0].float() * 0.1
    O1, O2, O3, O4 = (torch.empty(shape, dtype=torch.bfloat16, device=dev) for _ in range(4))
    R2 = torch.empty(shape, dtype=torch.float32, device=dev)
    say(f"narrow window B={B} H={H} L={L} d={d} w={w}")
    dfa.dfa_attn_full(gq, gk, gv, O1, w)
    dfa.dfa_attn_full_and_residual(gq, gk, gv, O2, R2, w)
    dfa.dfa_attn_window_plus_residual(gq, gk, gv, O3, Rres.to(dev), w)
    dfa.dfa_attn_window_plus_residual(gq, gk, gv, O4, None, w)
    torch.cuda.synchronize()
    check("full", O1, Of)
    check("refresh O", O2, Of)
    check("refresh R", R2, Of - Wd)
    check("window + R", O3, Wd + f64(Rres))
    check("window", O4, Wd)
    # Eq. 1 then Eq. 2: a reuse at drifted inputs adds the GPU's own residual;
    # the oracle chains its own residual
    dq, dk, dv = rand_qkv(shape, 6200 + L + w + d)
    q1, k1, v1 = ((x.float() + 0.05 * y.float()).to(torch.bfloat16) for x, y in zip((q, k, v), (dq, dk, dv)))
    O5 = torch.empty(shape, dtype=torch.bfloat16, device=dev)
    dfa.dfa_attn_window_plus_residual(q1.to(dev), k1.to(dev), v1.to(dev), O5, R2, w)
    torch.cuda.synchronize()
    check("reuse after refresh", O5, orc.wars_reuse(f64(q1), f64(k1), f64(v1), Of - Wd, w))


@pytest.mark.parametrize("B,H,L,d", [(1, 2, 333, 72), (1, 2, 200, 64), (3, 2, 16, 72)])
def test_extreme_half_widths(B, H, L, d):
    """Half-widths at and far beyond the sequence (up to the largest int):
    a band that covers every key gives the window attention of full attention
    and a residual of exactly zero; one key short of that it is a true band."""
    dev = torch.device("cuda")
    shape = (B, H, L, d)
    q, k, v = rand_qkv(shape, 900 + L + d)
    gq, gk, gv = (t.to(dev) for t in (q, k, v))
    Qd, Kd, Vd = f64(q), f64(k), f64(v)
    Of = orc.attn_full(Qd, Kd, Vd)
    for w in [L - 2, L - 1, L, 1 << 30, (1 << 31) - 1]:
        say(f"extreme half-width B={B} H={H} L={L} d={d} w={w}")
        O1, O2 = (torch.empty(shape, dtype=torch.bfloat16, device=dev) for _ in range(2))
        R = torch.full(shape, 7.0, dtype=torch.float32, device=dev)
        dfa.dfa_attn_window_plus_residual(gq, gk, gv, O1, None, w)
        dfa.dfa_attn_full_and_residual(gq, gk, gv, O2, R, w)
        torch.cuda.synchronize()
        check(f"window w={w}", O1, orc.attn_window(Qd, Kd, Vd, w))
        check(f"refresh O w={w}", O2, Of)
        if w >= L - 1:
            assert torch.count_nonzero(R).item() == 0, f"w={w}: R must be exactly zero"
        else:
            check(f"refresh R w={w}", R, Of - orc.attn_window(Qd, Kd, Vd, w))


def test_window_without_residual_and_determinism():
    dev = torch.device("cuda")
    shape = (2, 3, 700, 72)
    q, k, v = rand_qkv(shape, 42)
    gq, gk, gv = (t.to(dev) for t in (q, k, v))
    O = torch.empty(shape, dtype=torch.bfloat16, device=dev)
    say("window (no residual) L=700 w=87")
    dfa.dfa_attn_window_plus_residual(gq, gk, gv, O, None, 87)
    torch.cuda.synchronize()
    check("window", O, orc.attn_window(f64(q), f64(k), f64(v), 87))
    O_a, R_a = torch.empty_like(O), torch.empty(shape, dtype=torch.float32, device=dev)
    O_b, R_b = torch.empty_like(O), torch.empty_like(R_a)
    dfa.dfa_attn_full_and_residual(gq, gk, gv, O_a, R_a, 87)
    dfa.dfa_attn_full_and_residual(gq, gk, gv, O_b, R_b, 87)
    torch.cuda.synchronize()
    assert torch.equal(O_a, O_b) and torch.equal(R_a, R_b), "refresh must be deterministic"


def test_zero_drift_refresh_then_reuse():
    """Eq. 1 then Eq. 2 at unchanged inputs rebuilds the full output."""
    dev = torch.device("cuda")
    shape = (2, 2, 512, 72)
    q, k, v = (t.to(dev) for t in rand_qkv(shape, 5))
    O, O2, Of = (torch.empty(shape, dtype=torch.bfloat16, device=dev) for _ in range(3))
    R = torch.empty(shape, dtype=torch.float32, device=dev)
    say("zero drift L=512 w=64")
    dfa.dfa_attn_full_and_residual(q, k, v, O, R, 64)
    dfa.dfa_attn_window_plus_residual(q, k, v, O2, R, 64)
    dfa.dfa_attn_full(q, k, v, Of)
    torch.cuda.synchronize()
    # refresh sums two accumulators (in / out of the band): same value as full
    # attention up to rounding order
    assert float((O.float() - Of.float()).abs().max()) <= 2 ** -8
    err = (O2.float() - O.float()).abs()
    assert float(err.max()) <= 2 ** -7 and float(err.mean()) <= 1e-3


def test_tiny_three_step_check():
    """One layer, B=2 (a CFG pair), H=2, L=256, d=64, w=16; step 0 refresh,
    steps 1-2 reuse with 0.05 drift per step; fp32 masters rounded to bf16."""
    cfg = inputs.CONFIGS["tiny"]
    dev = torch.device("cuda")
    shape = (cfg.B, cfg.H, cfg.L, cfg.d)
    codes = [dfa.WARS_REFRESH, dfa.WARS_REUSE, dfa.WARS_REUSE]
    gen = inputs.DriftingQKV(cfg.cfg_id, 0, shape, cfg.drift)
    O, Oc = (torch.empty(shape, dtype=torch.bfloat16, device=dev) for _ in range(2))
    R = torch.empty(shape, dtype=torch.float32, device=dev)
    cache = orc.LayerCache()
    for t, c in enumerate(codes):
        q, k, v = gen.advance()
        say(f"tiny step {t} code {dfa.CODE_NAMES[c]}")
        dfa.dfa_plan_step(c, q.to(dev), k.to(dev), v.to(dev), O, R, Oc, cfg.w)
        torch.cuda.synchronize()
        ref = orc.plan_step(c, f64(q), f64(k), f64(v), cache, cfg.w)
        check(f"tiny O step {t}", O, ref)
        assert torch.equal(O, Oc)
        if c == dfa.WARS_REFRESH:
            check("tiny R", R, cache.R)
        # secondary number: the same step against the un-rounded fp32 masters
        masters = [m.astype(np.float64) for m in gen.master]
        if t == 0:
            ref32 = orc.attn_full(*masters)
            e32 = float(np.abs(f64(O) - ref32).max())
            say(f"tiny step 0 vs fp32 masters: max abs {e32:.3e}")


HALF_BATCH = (dfa.ASC_REUSE, dfa.WARS_ASC_REFRESH, dfa.WARS_ASC_REUSE)
# a legal sequence that runs every plan code, including a combined reuse fed
# by a whole-batch refresh and one fed by a conditional-half refresh
MIXED_CODES = [dfa.WARS_REFRESH, dfa.WARS_REUSE, dfa.WARS_ASC_REUSE, dfa.AST_REUSE, dfa.WARS_ASC_REFRESH,
               dfa.WARS_ASC_REUSE, dfa.ASC_REUSE, dfa.FULL, dfa.AST_REUSE, dfa.WARS_REFRESH, dfa.WARS_REUSE,
               dfa.WARS_ASC_REUSE]


def run_plan(cfg_key, layers, n_steps, n_rows=None, alias_cache=(), codes=None):
    cfg = inputs.CONFIGS[cfg_key]
    dev = torch.device("cuda")
    shape = (cfg.B, cfg.H, cfg.L, cfg.d)
    half = cfg.B // 2
    if codes is None:
        code, r_src, o_src = dfa.dfa_plan_make(cfg.plan_seed, cfg.n_layers, cfg.n_steps, cfg.refresh_every, cfg.B)
        ref_plan = orc.plan_make(cfg.plan_seed, cfg.n_layers, cfg.n_steps, cfg.refresh_every, cfg.B)
        for a, b in zip((code, r_src, o_src), ref_plan):
            assert np.array_equal(a, b)
    else:
        code, r_src, o_src = orc.fixed_plan(codes, n_layers=max(layers) + 1)
    rows = None if n_rows is None else inputs.sample_rows(cfg.L, n_rows, cfg.cfg_id)
    seen = set()
    for layer in layers:
        gen = inputs.DriftingQKV(cfg.cfg_id, layer, shape, cfg.drift)
        O = Guarded(shape, dev).t
        Rg = Guarded(shape, dev, torch.float32)
        R = Rg.t
        Oc = O if layer in alias_cache else Guarded(shape, dev).t
        cache = orc.LayerCache()
        outputs = {}
        for t in range(n_steps):
            q, k, v = gen.advance()
            c = int(code[t, layer])
            seen.add(c)
            say(f"{cfg_key} layer {layer} step {t} code {dfa.CODE_NAMES[c]}")
            if t == 0:
                R_before = R.cpu()
            if c == dfa.AST_REUSE:
                dfa.dfa_plan_step(c, None, None, None, O, R, Oc, cfg.w)
            else:
                dfa.dfa_plan_step(c, q.to(dev), k.to(dev), v.to(dev), O, R, Oc, cfg.w)
            torch.cuda.synchronize()
            Qd, Kd, Vd = f64(q), f64(k), f64(v)
            if rows is None:
                ref = orc.plan_step(c, Qd, Kd, Vd, cache, cfg.w)
            else:
                ref = orc.plan_step_rows(c, Qd, Kd, Vd, rows, cache, cfg.w)
            got = O.cpu()
            check(f"{cfg_key} l{layer} t{t} O", got, ref, rows)
            if c == dfa.WARS_REFRESH:
                check(f"{cfg_key} l{layer} t{t} R", R, cache.R, rows)
            if c == dfa.WARS_ASC_REFRESH:
                check(f"{cfg_key} l{layer} t{t} R[cond]", R[:half], cache.R, rows)
                assert torch.equal(R[half:].cpu(), R_before[half:]), "a half-batch refresh must leave R[uncond]"
            if c == dfa.AST_REUSE:
                assert torch.equal(got, outputs[int(o_src[t, layer])]), "AST must return the cached step bitwise"
            else:
                outputs[t] = got
                assert torch.equal(Oc.cpu(), got), "computed steps must refresh the cache"
            if c in HALF_BATCH:
                assert torch.equal(got[:half], got[half:]), "CFG-shared halves must be bit-identical"
            R_before = R.cpu()
        assert Rg.guards_intact(), "write outside R"
    return seen


def test_plan_dit256():
    seen = run_plan("dit256", layers=[0, 1], n_steps=50, alias_cache={1})
    assert seen == {0, 1, 2, 3, 4}


def test_plan_dit512_sampled():
    run_plan("dit512", layers=[3], n_steps=50, n_rows=96)


def test_plan_dit512_all_rows():
    """The first steps of a DiT-XL/2 512 layer, every query row of every
    (batch, head) against the whole-sequence oracle."""
    seen = run_plan("dit512", layers=[0], n_steps=8)
    assert {dfa.WARS_REFRESH, dfa.WARS_REUSE} <= seen


def test_plan_pixart1k_sampled():
    run_plan("pixart1k", layers=[0, 5], n_steps=20, n_rows=128, alias_cache={5})


def test_plan_pixart2k_sampled():
    """Every step of two PixArt-Sigma 2K layers (refresh every 4 steps)."""
    seen = run_plan("pixart2k", layers=[2, 11], n_steps=20, n_rows=64, alias_cache={11})
    assert {dfa.WARS_REFRESH, dfa.WARS_REUSE} <= seen


def test_plan_mixed_codes_dit256():
    """Every plan code, including WA-RS + ASC after both kinds of refresh."""
    seen = run_plan("dit256", layers=[0, 1], n_steps=len(MIXED_CODES), alias_cache={1}, codes=MIXED_CODES)
    assert seen == set(dfa.CODE_NAMES)


def test_plan_mixed_codes_pixart2k_sampled():
    run_plan("pixart2k", layers=[4], n_steps=len(MIXED_CODES), n_rows=48, codes=MIXED_CODES)


def test_wars_asc_odd_shapes():
    """WA-RS + ASC on ragged tiles and degenerate bands (B = 4: two CFG pairs)."""
    dev = torch.device("cuda")
    for (B, H, L, d, w) in ((4, 1, 77, 72, 5), (2, 2, 129, 64, 0), (4, 2, 300, 72, 299), (2, 1, 1, 72, 0),
                            (4, 3, 16, 72, 2), (2, 1, 29, 64, 28)):
        shape = (B, H, L, d)
        say(f"wars+asc B={B} H={H} L={L} d={d} w={w}")
        q0, k0, v0 = rand_qkv(shape, 300 + L + w)
        q1, k1, v1 = (x + 0.05 * y for x, y in zip((q0, k0, v0), rand_qkv(shape, 400 + L)))
        O, Oc = Guarded(shape, dev), Guarded(shape, dev)
        Rg = Guarded(shape, dev, torch.float32)
        Rg.t.fill_(-7.0)
        cache = orc.LayerCache()
        for c, (q, k, v) in ((dfa.WARS_ASC_REFRESH, (q0, k0, v0)), (dfa.WARS_ASC_REUSE, (q1, k1, v1))):
            dfa.dfa_plan_step(c, q.to(dev), k.to(dev), v.to(dev), O.t, Rg.t, Oc.t, w)
            torch.cuda.synchronize()
            ref = orc.plan_step(c, f64(q), f64(k), f64(v), cache, w)
            check(f"wars+asc {dfa.CODE_NAMES[c]} O", O.t, ref)
            got = O.t.cpu()
            assert torch.equal(got[: B // 2], got[B // 2:]) and torch.equal(Oc.t.cpu(), got)
        check("wars+asc R[cond]", Rg.t[: B // 2], cache.R)
        assert bool(torch.all(Rg.t[B // 2:] == -7.0)), "R[uncond] must stay untouched"
        if w >= L - 1:
            assert not torch.any(Rg.t[: B // 2] != 0), "w >= L-1 must give R == 0 exactly"
        for g in (O, Oc, Rg):
            assert g.guards_intact(), "write outside an output tensor"


def test_checkpoint_resume_bit_exact():
    """Stop a plan run after step k, move the layer's caches (R, Ocache) to the
    host and back into fresh buffers, continue: every later output equals the
    uninterrupted run bit for bit."""
    cfg = inputs.CONFIGS["dit256"]
    dev = torch.device("cuda")
    shape = (cfg.B, cfg.H, cfg.L, cfg.d)
    steps = [inputs.bf16_qkv(cfg.cfg_id, 0, t, shape) for t in range(len(MIXED_CODES))]
    steps = [tuple(x.to(dev) for x in qkv) for qkv in steps]

    def fresh():
        return (torch.zeros(shape, dtype=torch.bfloat16, device=dev),
                torch.zeros(shape, dtype=torch.float32, device=dev),
                torch.zeros(shape, dtype=torch.bfloat16, device=dev))

    def run(t0, t1, O, R, Oc):
        outs = []
        for t in range(t0, t1):
            c = MIXED_CODES[t]
            q, k, v = steps[t] if c != dfa.AST_REUSE else (None, None, None)
            dfa.dfa_plan_step(c, q, k, v, O, R, Oc, cfg.w)
            outs.append(O.clone())
        torch.cuda.synchronize()
        return outs

    say("checkpoint/resume: uninterrupted run")
    ref = run(0, len(MIXED_CODES), *fresh())
    for k in (3, 5, 9):
        say(f"checkpoint/resume: cut after step {k - 1}")
        O, R, Oc = fresh()
        run(0, k, O, R, Oc)
        saved = (R.cpu(), Oc.cpu())
        del O, R, Oc
        O2, R2, Oc2 = fresh()
        R2.copy_(saved[0])
        Oc2.copy_(saved[1])
        outs = run(k, len(MIXED_CODES), O2, R2, Oc2)
        for t, got in zip(range(k, len(MIXED_CODES)), outs):
            assert torch.equal(got, ref[t]), f"resumed run differs at step {t} ({dfa.CODE_NAMES[MIXED_CODES[t]]})"


@pytest.mark.parametrize("key,n_rows", [("opensora_spatial", 64), ("opensora_temporal", None)])
def test_video_shapes(key, n_rows):
    """Open-Sora-shaped spatial (405 tokens per frame) and temporal (16
    frames) attention through every plan code, CFG pairs batch-major."""
    run_plan(key, layers=[0], n_steps=len(MIXED_CODES), n_rows=n_rows, codes=MIXED_CODES)
