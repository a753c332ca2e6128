"""Seeded tensor generators (no method arithmetic here, only random draws)."""
from __future__ import annotations

import math

import numpy as np
import torch

from .configs import MoEConfig

# tensor ids inside a seed tuple
_X, _WG, _RANK, _GATE, _UP, _DOWN, _PW1, _PW2 = range(8)


def tensor_seed(cfg: MoEConfig, layer: int, expert: int, tensor: int, base: int = 0) -> int:
    """64-bit seed for one tensor, from SeedSequence([base, workload, layer, expert, tensor])."""
    ss = np.random.SeedSequence([base, cfg.cid, layer, expert, tensor])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & 0x7FFF_FFFF_FFFF_FFFF)


def _randn(shape, seed: int, device, std: float = 1.0):
    dev = torch.device(device)
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    t = torch.randn(shape, generator=g, device=dev, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t


def _act(t: torch.Tensor, cfg: MoEConfig) -> torch.Tensor:
    return t if cfg.act == "f32" else t.to(torch.bfloat16)


def activations(cfg: MoEConfig, layer: int = 0, device="cpu", T: int | None = None, base: int = 0):
    """x [T][C] ~ N(0, 1) in the workload's activation dtype (bf16 rounding by torch)."""
    T = cfg.T if T is None else T
    return _act(_randn((T, cfg.C), tensor_seed(cfg, layer, 0, _X, base), device), cfg)


def router_weights(cfg: MoEConfig, layer: int = 0, device="cpu"):
    """Router matrix Wg [E][C] ~ N(0, 1/C) in the activation dtype."""
    std = 1.0 / math.sqrt(cfg.C)
    return _act(_randn((cfg.E, cfg.C), tensor_seed(cfg, layer, 0, _WG), device, std), cfg)


def _layer_rank(cfg: MoEConfig, layer: int) -> np.ndarray:
    """Popularity rank of each expert; stacked layers get a seeded shuffle per layer."""
    if cfg.layers <= 1:
        return np.arange(cfg.E)
    rng = np.random.Generator(np.random.PCG64(tensor_seed(cfg, layer, 0, _RANK)))
    return rng.permutation(cfg.E)


def router_bias(cfg: MoEConfig, layer: int = 0):
    """Zipf-skewed router bias b_e = -s * ln(rank(e) + 1) (fp32 [E]), or None."""
    if cfg.zipf_s == 0.0:
        return None
    rank = _layer_rank(cfg, layer)
    b = np.array([-cfg.zipf_s * math.log(r + 1.0) for r in rank], dtype=np.float32)
    return torch.from_numpy(b)


def resident_experts(cfg: MoEConfig, layer: int = 0):
    """Experts resident on the GPU for a layer: the `resident` most popular ones (all if 0)."""
    if cfg.resident <= 0:
        return list(range(cfg.E))
    rank = _layer_rank(cfg, layer)
    return sorted(int(e) for e in np.argsort(rank, kind="stable")[: cfg.resident])


def expert_weights(cfg: MoEConfig, layer: int, expert: int, device="cpu"):
    """fp32 master weights of one expert (routed 0..E-1, shared E..E+S-1).

    Returns (w_gate [R][C], w_up [R][C], w_down [C][R]), each ~ N(0, w_std^2).
    """
    s = cfg.w_std
    wg = _randn((cfg.R, cfg.C), tensor_seed(cfg, layer, expert, _GATE), device, s)
    wu = _randn((cfg.R, cfg.C), tensor_seed(cfg, layer, expert, _UP), device, s)
    wd = _randn((cfg.C, cfg.R), tensor_seed(cfg, layer, expert, _DOWN), device, s)
    return wg, wu, wd


def predictor_weights(cfg: MoEConfig, layer: int, device="cpu"):
    """Predictor MLP C -> P -> E: W1 [P][C] ~ N(0, 1/C), W2 [E][P] ~ N(0, 1/P), bf16; zero biases."""
    P = cfg.pred_hidden
    w1 = _randn((P, cfg.C), tensor_seed(cfg, layer, 0, _PW1), device, 1.0 / math.sqrt(cfg.C))
    w2 = _randn((cfg.E, P), tensor_seed(cfg, layer, 0, _PW2), device, 1.0 / math.sqrt(P))
    b1 = torch.zeros(P, dtype=torch.float32, device=device)
    b2 = torch.zeros(cfg.E, dtype=torch.float32, device=device)
    return w1.to(torch.bfloat16), b1, w2.to(torch.bfloat16), b2


def drift_bias(cfg: MoEConfig, layer: int, epoch: int):
    """Router bias of a workload whose expert popularity drifts: the Zipf-ranked
    bias -s * ln(rank(e) + 1) with a seeded rank permutation per (layer, epoch)."""
    rng = np.random.Generator(np.random.PCG64(tensor_seed(cfg, layer, epoch, _RANK, base=7)))
    rank = rng.permutation(cfg.E)
    b = np.array([-cfg.zipf_s * math.log(r + 1.0) for r in rank], dtype=np.float32)
    return torch.from_numpy(b)


def drift_hot(cfg: MoEConfig, layer: int, epoch: int, n: int):
    """The n most popular experts of a drifting layer in one epoch."""
    rng = np.random.Generator(np.random.PCG64(tensor_seed(cfg, layer, epoch, _RANK, base=7)))
    rank = rng.permutation(cfg.E)
    return sorted(int(e) for e in np.argsort(rank, kind="stable")[:n])
