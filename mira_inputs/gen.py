"""Seeded tensor generators (no method arithmetic here, only random draws)."""
from __future__ import annotations

import math

import numpy as np
import torch

from .configs import MoEConfig

# tensor ids inside a seed tuple
_X, _WG, _RANK, _GATE, _UP, _DOWN, _PW1, _PW2, _ROUTE, _MIX = range(10)


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


_MIX_MATS = (("wah", "Pa", "C"), ("wal", "Pa", "E"), ("wa2", "N", "Pa"), ("whq", "Ph", "E"),
             ("whu", "Ph", "E"), ("wh2", "N", "Ph"), ("gh", None, "C"), ("gl", None, "E"),
             ("gq", None, "E"), ("gu", None, "E"))
_MIX_BIAS = (("ba1", "Pa"), ("ba2", "N"), ("bh1", "Ph"), ("bh2", "N"))


def mixture_weights(cfg: MoEConfig, layer: int, act_hidden: int, hist_hidden: int,
                    n_out: int | None = None, device="cpu"):
    """Synthetic MixtureHead weights for a source layer with cfg.E experts.

    Matrices and gate vectors are bf16 ~ N(0, 1/fan_in) (fan_in = their
    column count; the gate's over all of C + 3E features), biases fp32
    ~ N(0, 0.1^2), the gate bias a float ~ N(0, 0.25^2).  Returns a dict keyed
    like the C struct's fields."""
    dims = {"C": cfg.C, "E": cfg.E, "Pa": act_hidden, "Ph": hist_hidden,
            "N": cfg.E if n_out is None else n_out}
    out = {}
    for j, (name, rows, cols) in enumerate(_MIX_MATS):
        fan = dims[cols] if rows else cfg.C + 3 * cfg.E
        shape = (dims[rows], dims[cols]) if rows else (dims[cols],)
        t = _randn(shape, tensor_seed(cfg, layer, j, _MIX), device, 1.0 / math.sqrt(fan))
        out[name] = t.to(torch.bfloat16)
    for j, (name, size) in enumerate(_MIX_BIAS):
        out[name] = _randn((dims[size],), tensor_seed(cfg, layer, 100 + j, _MIX), device, 0.1)
    out["bg"] = float(_randn((1,), tensor_seed(cfg, layer, 200, _MIX), "cpu", 0.25)[0])
    return out


def routing_sample(cfg: MoEConfig, layer: int, T: int | None = None):
    """A synthetic routing record of a source layer, on the host: logits [T][E]
    fp32 ~ N(0, 1) and topk_idx [T][k] int32, k distinct experts per token
    drawn without replacement with Zipf(cfg.zipf_s) popularity over a seeded
    ranking (uniform if zipf_s is 0)."""
    T = cfg.T if T is None else T
    logits = _randn((T, cfg.E), tensor_seed(cfg, layer, 0, _ROUTE), "cpu")
    rng = np.random.Generator(np.random.PCG64(tensor_seed(cfg, layer, 1, _ROUTE)))
    rank = rng.permutation(cfg.E)
    p = (rank + 1.0) ** -cfg.zipf_s
    p /= p.sum()
    idx = np.stack([rng.choice(cfg.E, size=cfg.k, replace=False, p=p) for _ in range(T)]) if T else \
        np.zeros((0, cfg.k), dtype=np.int64)
    return logits, torch.from_numpy(idx.astype(np.int32))
