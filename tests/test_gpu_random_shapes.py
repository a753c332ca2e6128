"""A seeded sweep of random small layer shapes through the whole layer call
on the GPU, against the oracle: hidden size and ffn (multiples of 64, or of
128 for the INT4 variant), routed and shared expert counts, top-k, token
counts on both sides of the decode limit (and a sweep of one-token calls),
bf16 and fp32 activations, with and without a router bias.  Every case checks routing bit-exactly and every
output row within the error bars (run_and_check)."""
import numpy as np
import pytest

from gpu_layer import Layer, decode_rel_floor, run_and_check
from mira_inputs import MoEConfig

pytestmark = pytest.mark.gpu


def _cases(seed, n, int4, one_token=False):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        step = 128 if int4 else 64
        C = step * int(rng.integers(1, 9 if one_token else 5))
        R = step * int(rng.integers(1, 49 if one_token else 7))
        E = int(rng.choice([1, 2, 3, 5, 8, 13, 32, 64]))
        S = int(rng.integers(0, 3))
        k = int(rng.integers(1, min(E, 8) + 1))
        if one_token:
            T = 1
        else:
            T = int(rng.integers(1, 17)) if (int4 or rng.random() < 0.5) else int(rng.integers(17, 301))
        act = "f32" if rng.random() < 0.3 else "bf16"
        zipf = float(rng.choice([0.0, 1.0, 1.2]))
        tag = ("1" if one_token else "") + ("4" if int4 else "8")
        cfg = MoEConfig(f"rand{tag}_{i}", 200 + i + (100 if int4 else 0) + (400 if one_token else 0), T=T, C=C, E=E,
                        k=k, R=R, S=S, act=act, zipf_s=zipf)
        out.append(pytest.param(cfg, id=f"C{C}-R{R}-E{E}-S{S}-k{k}-T{T}-{act}"))
    return out


@pytest.mark.parametrize("cfg", _cases(7, 24, int4=False))
def test_random_shape_int8(mira, cfg):
    res, errs, _, _ = run_and_check(Layer(cfg))
    if cfg.T <= mira.MIRA_DECODE_MAX_TOKENS:
        assert errs[0] < decode_rel_floor(cfg.T), errs


@pytest.mark.parametrize("cfg", _cases(8, 8, int4=True))
def test_random_shape_int4(mira, cfg):
    res, errs, _, _ = run_and_check(Layer(cfg, fmt="int4"))
    assert errs[0] < decode_rel_floor(cfg.T), errs


# One-token calls take their own kernels (the tile split of gate/up over the
# CUs, per-tile H' exponents in the down kernel): a sweep of their own with
# ffn up to 48 blocks, so tile counts from a handful to a few thousand,
# ragged last workgroups and several wave counts per workgroup come up.
@pytest.mark.parametrize("cfg", _cases(9, 12, int4=False, one_token=True))
def test_random_one_token_int8(mira, cfg):
    res, errs, _, _ = run_and_check(Layer(cfg))
    assert errs[0] < decode_rel_floor(1), errs


@pytest.mark.parametrize("cfg", _cases(10, 8, int4=True, one_token=True))
def test_random_one_token_int4(mira, cfg):
    res, errs, _, _ = run_and_check(Layer(cfg, fmt="int4"))
    assert errs[0] < decode_rel_floor(1), errs
