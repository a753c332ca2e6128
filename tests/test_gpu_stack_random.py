"""A seeded sweep of random expert-stack settings (sections IV-C to IV-F):
layer count, experts per layer, top-k, resident experts, STAGE capacity,
small or large VRAM mode, lookahead, prefetch width, MLP or MixtureHead,
the rebalancer on or off, and the staging mode of each step.  Whatever the
runtime serves from HOT, STAGE or a demand copy, every layer's output must
match the oracle on the layer's input, and the counters must add up."""
import numpy as np
import pytest

from gpu_layer import assert_ffn_close
from mira_inputs import MoEConfig
from test_gpu_stack import build, oracle_layer, run, true_routing

pytestmark = pytest.mark.gpu


def _cases(seed, n):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        E = int(rng.choice([4, 6, 8]))
        k = int(rng.integers(1, 3))
        group = int(rng.choice([4, 8]))
        T = group * int(rng.integers(1, 3))
        layers = int(rng.integers(3, 7))
        resident = int(rng.integers(1, E))
        need = min(E - resident, T * k)  # non-HOT experts one layer can select
        n_stage = need + int(rng.integers(0, 4))
        kw = dict(vram_mode=str(rng.choice(["large", "small"])), head=str(rng.choice(["mlp", "mixture"])),
                  lookahead=int(rng.integers(1, 3)), stage_per_layer=int(rng.integers(1, 4)),
                  rebalance=bool(rng.random() < 0.5))
        cfg = MoEConfig(f"stack_rand_{i}", 400 + i, T=T, C=128, E=E, k=k, R=128, zipf_s=1.0, layers=layers,
                        resident=resident, pred_hidden=32, pred_group=group)
        ident = (f"L{layers}-E{E}-k{k}-T{T}-hot{resident}-stage{n_stage}-{kw['vram_mode']}-{kw['head']}"
                 f"-la{kw['lookahead']}-w{kw['stage_per_layer']}{'-rb' if kw['rebalance'] else ''}")
        out.append(pytest.param(cfg, n_stage, kw, id=ident))
    return out


@pytest.mark.parametrize("cfg,n_stage,kw", _cases(11, 12))
def test_random_stack_settings_match_oracle(mira, cfg, n_stage, kw):
    from paper_2609_38090_amd.policy import RebalanceConfig, Rebalancer
    rb = Rebalancer(RebalanceConfig(interval=cfg.T * 2, max_swaps=1, probation=1)) if kw["rebalance"] else None
    st, blobs = build(mira, cfg, n_stage, host_all=rb is not None, rebalancer=rb, head=kw["head"],
                      vram_mode=kw["vram_mode"], lookahead=kw["lookahead"],
                      stage_per_layer=kw["stage_per_layer"])
    true_idx = true_routing(mira, st, cfg)
    for step, mode in enumerate(("demand", "oracle", "predict", "predict")):
        outs, stats = run(st, mode, true_idx=true_idx)
        for l in range(cfg.layers):
            assert_ffn_close(outs[l], oracle_layer(st, cfg, blobs, l)["out"], f"step {step} ({mode}) layer {l}")
        # every selected (layer, expert) pair was served exactly once
        selected = sum(len(set(true_idx[l].reshape(-1).tolist())) for l in range(cfg.layers))
        assert stats.hot_hits + stats.stage_hits + stats.misses == selected, (step, mode)
        assert stats.hot_tokens + stats.stage_tokens + stats.cpu_tokens == cfg.layers * cfg.T * cfg.k
        if mode == "demand":
            assert stats.prefetches == stats.prefetch_cached == stats.prefetch_declined == 0
