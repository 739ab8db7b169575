"""Seeded synthetic inputs for the attention hot path.

This module only draws random numbers and rounds them to bf16; it contains
none of the attention method's arithmetic.  Both sides of every parity check
(the HIP library and the fp64 oracle) receive the same bf16 values from here.

Recipe (stands in for the Q/K/V of a trained DiT; no dataset or weights):
  * per (config, layer, tensor) an fp32 master X_0 ~ N(0, 1), drawn from
    numpy PCG64 seeded with SeedSequence([240608552, cfg, layer, 0, tensor]),
    tensor 0/1/2 = Q/K/V;
  * drift per step: X_t = X_{t-1} + drift * N(0, 1), the step-t normals drawn
    from SeedSequence([240608552, cfg, layer, t, tensor]);
  * each use rounds X_t to bf16 (round to nearest even).
For bench-scale tensors ``device_qkv`` draws on the device with torch's
seeded generator instead (same distribution, different stream).

Attention-module inputs (random weights stand in for a trained DiT):
  * hidden states X [B, L, C], C = H * d, follow the same drifting recipe
    (tensor index 3);
  * W_qkv [3C, C] and W_o [C, C] are N(0, 1/C) rounded to bf16, the biases
    0.1 * N(0, 1) in fp32, from SeedSequence([240608552, 77, seed, k]).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

SEED_BASE = 240608552


@dataclass(frozen=True)
class AttnConfig:
    """One attention workload: shapes, band half-width and plan schedule."""
    name: str
    cfg_id: int
    B: int
    H: int
    L: int
    d: int
    w: int
    n_layers: int
    n_steps: int
    refresh_every: int
    drift: float = 0.05
    fp32_inputs: bool = False   # the tiny check draws fp32 masters

    @property
    def plan_seed(self) -> int:
        return SEED_BASE + self.cfg_id


# The five workloads: a tiny three-step check and four DiT / PixArt-Sigma
# shaped attention layers (L = (resolution / 16)^2 tokens, H = 16, d = 72).
CONFIGS = {
    "tiny": AttnConfig("tiny_wars_check", 1, B=2, H=2, L=256, d=64, w=16,
                       n_layers=1, n_steps=3, refresh_every=0, fp32_inputs=True),
    "dit256": AttnConfig("dit_xl2_256px", 2, B=8, H=16, L=256, d=72, w=32,
                         n_layers=28, n_steps=50, refresh_every=0),
    "dit512": AttnConfig("dit_xl2_512px", 3, B=8, H=16, L=1024, d=72, w=128,
                         n_layers=28, n_steps=50, refresh_every=0),
    "pixart1k": AttnConfig("pixart_sigma_1024px", 4, B=2, H=16, L=4096, d=72, w=512,
                           n_layers=28, n_steps=20, refresh_every=4),
    "pixart2k": AttnConfig("pixart_sigma_2048px", 5, B=2, H=16, L=16384, d=72, w=2048,
                           n_layers=28, n_steps=20, refresh_every=4),
    # Open-Sora V1.1 at 240p with 16 frames (STDiT: hidden 1152 = 16 heads x 72).
    # The paper gives no attention shapes; read here as 240 x 426 frames, an 8x
    # VAE and 2 x 2 patches: 15 x 27 = 405 tokens per frame.  Spatial attention
    # runs within each frame (batch = CFG pair x 16 frames, CFG-major), temporal
    # attention across the 16 frames of each token (batch = CFG pair x 405).
    "opensora_spatial": AttnConfig("opensora_v1.1_240p_16f_spatial", 6, B=32, H=16, L=405, d=72, w=50,
                                   n_layers=28, n_steps=20, refresh_every=0),
    "opensora_temporal": AttnConfig("opensora_v1.1_240p_16f_temporal", 7, B=810, H=16, L=16, d=72, w=2,
                                    n_layers=28, n_steps=20, refresh_every=0),
}


def _normals(cfg_id: int, layer: int, step: int, tensor: int, shape) -> np.ndarray:
    ss = np.random.SeedSequence([SEED_BASE, cfg_id, layer, step, tensor])
    return np.random.Generator(np.random.PCG64(ss)).standard_normal(shape, dtype=np.float32)


def master_qkv(cfg_id: int, layer: int, step: int, shape, drift: float = 0.05):
    """fp32 masters (Q, K, V) of one layer at one step (random walk over steps)."""
    out = []
    for tensor in range(3):
        x = _normals(cfg_id, layer, 0, tensor, shape)
        for t in range(1, step + 1):
            x = x + np.float32(drift) * _normals(cfg_id, layer, t, tensor, shape)
        out.append(x)
    return tuple(out)


class DriftingQKV:
    """Iterates the (Q, K, V) of one layer over steps 0, 1, 2, ... keeping the
    fp32 masters, so step t costs one draw per tensor."""

    def __init__(self, cfg_id: int, layer: int, shape, drift: float = 0.05):
        self.cfg_id, self.layer, self.shape, self.drift = cfg_id, layer, tuple(shape), drift
        self.step = -1
        self.master = None

    def advance(self):
        self.step += 1
        t = self.step
        if t == 0:
            self.master = [_normals(self.cfg_id, self.layer, 0, i, self.shape) for i in range(3)]
        else:
            self.master = [m + np.float32(self.drift) * _normals(self.cfg_id, self.layer, t, i, self.shape)
                           for i, m in enumerate(self.master)]
        return to_bf16(self.master)


class DriftingX:
    """Hidden states [B, L, C] of one layer over steps 0, 1, 2, ... (fp32
    masters, random walk with the given drift), rounded to bf16 per use."""

    def __init__(self, cfg_id: int, layer: int, shape, drift: float = 0.05):
        self.cfg_id, self.layer, self.shape, self.drift = cfg_id, layer, tuple(shape), drift
        self.step = -1
        self.master = None

    def advance(self):
        self.step += 1
        z = _normals(self.cfg_id, self.layer, self.step, 3, self.shape)
        self.master = z if self.step == 0 else self.master + np.float32(self.drift) * z
        return to_bf16([self.master])[0]


def surrogate_states(seed: int, B: int, L: int, C: int, n_steps: int, drift: float, cfg_gap: float = 0.1):
    """Hidden states [B, L, C] bf16 of a surrogate model over n_steps steps.
    The conditional half drifts by `drift` per step (DriftingX recipe); the
    unconditional partner of entry b is entry b plus cfg_gap times an
    independent drifting draw, so the CFG halves are close but not equal."""
    cond = DriftingX(seed, 0, (B, L, C), drift)
    other = DriftingX(seed, 1, (B, L, C), drift)
    half = B // 2
    out = []
    for _ in range(n_steps):
        a = as_f64(cond.advance())
        b = as_f64(other.advance())
        x = a.copy()
        x[half:] = a[:half] + cfg_gap * b[:half]
        out.append(torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16))
    return out


def module_weights(seed: int, H: int, d: int):
    """(W_qkv bf16 [3C, C], b_qkv fp32 [3C], W_o bf16 [C, C], b_o fp32 [C]) CPU tensors."""
    C = H * d

    def normals(k, shape):
        ss = np.random.SeedSequence([SEED_BASE, 77, seed, k])
        return np.random.Generator(np.random.PCG64(ss)).standard_normal(shape, dtype=np.float32)

    scale = np.float32(1.0 / np.sqrt(C))
    Wqkv = to_bf16([normals(0, (3 * C, C)) * scale])[0]
    Wo = to_bf16([normals(2, (C, C)) * scale])[0]
    bqkv = torch.from_numpy(np.float32(0.1) * normals(1, (3 * C,)))
    bo = torch.from_numpy(np.float32(0.1) * normals(3, (C,)))
    return Wqkv, bqkv, Wo, bo


def to_bf16(arrays):
    """Round fp32 arrays to bf16 (nearest even); returns CPU torch tensors."""
    return tuple(torch.from_numpy(np.ascontiguousarray(a)).to(torch.bfloat16) for a in arrays)


def as_f64(t: torch.Tensor) -> np.ndarray:
    """The exact float64 value of a bf16 (or any) tensor, on the host."""
    return t.detach().to("cpu", torch.float64).numpy()


def bf16_qkv(cfg_id: int, layer: int, step: int, shape, drift: float = 0.05):
    """bf16 (Q, K, V) CPU tensors of one layer at one step."""
    return to_bf16(master_qkv(cfg_id, layer, step, shape, drift))


def device_qkv(seed: int, shape, device, n: int = 3):
    """Bench-scale inputs: n bf16 N(0, 1) tensors drawn on ``device`` from a
    torch generator seeded with ``seed``."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return tuple(torch.randn(shape, generator=g, device=device, dtype=torch.float32)
                 .to(torch.bfloat16) for _ in range(n))


def sample_rows(L: int, n: int, seed: int) -> np.ndarray:
    """A sorted seeded sample of n distinct query rows out of L, always
    including the first and last rows (the band's truncated edges)."""
    if n >= L:
        return np.arange(L)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_BASE, 99, L, n, seed])))
    inner = rng.choice(np.arange(1, L - 1), size=n - 2, replace=False)
    return np.sort(np.concatenate([[0, L - 1], inner])).astype(np.int64)
