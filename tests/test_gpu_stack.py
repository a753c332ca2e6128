"""A stack of MoE layers over HOT and STAGE slots (paper sections IV-C, IV-E,
IV-F): every layer's output must be the same whether an expert is served from
its HOT slot, a STAGE slot filled ahead of time or a demand copy, and must
match the oracle (each layer on its own seeded input)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_layer import EPS, assert_ffn_close
from mira_inputs import (MoEConfig, activations, expert_weights, predictor_weights, resident_experts,
                         router_bias, router_weights)

pytestmark = pytest.mark.gpu

SMALL_STACK = MoEConfig("small_stack", 104, T=8, C=128, E=8, k=2, R=192, zipf_s=1.2, layers=5, resident=4,
                        pred_hidden=32, pred_group=8)


def build(mira, cfg, n_stage):
    from paper_2609_38090_amd.stack import ExpertStack, LayerData
    stride = mira.mira_packed_expert_bytes(cfg.C, cfg.R)
    layers, blobs = [], {}
    for l in range(cfg.layers):
        b = router_bias(cfg, l)
        pred = tuple(t.cuda() for t in predictor_weights(cfg, l, "cpu")) if l + 2 < cfg.layers else None
        layers.append(LayerData(x=activations(cfg, l, "cuda"), w_router=router_weights(cfg, l, "cuda"),
                                bias=None if b is None else b.cuda(), hot=resident_experts(cfg, l), pred=pred))
    shape = mira.MoEShape(cfg.C, cfg.R, cfg.E, cfg.k, cfg.S, mira.MIRA_BF16, 0)
    ps = mira.PredShape(cfg.C, cfg.pred_hidden, cfg.E, cfg.pred_group, mira.MIRA_BF16)
    st = ExpertStack(shape, cfg.T, layers, stride, n_stage=n_stage, pred_shape=ps)
    pack_shape = mira.MoEShape(cfg.C, cfg.R, 1, 1)
    for l, ld in enumerate(layers):
        for e in range(cfg.E):
            w = [np.ascontiguousarray(t.numpy()) for t in expert_weights(cfg, l, e, "cpu")]
            blobs[l, e] = oracle.pack_expert(*w, eps=EPS)  # the oracle's own packing, for the reference
            pinned = torch.zeros(stride, dtype=torch.uint8).pin_memory()
            mira.mira_pack_experts(pack_shape, 1, mira.MIRA_F32, w[0].ctypes.data, w[1].ctypes.data,
                                   w[2].ctypes.data, EPS, pinned, stride, 0)
            if e in st.hot_slot[l]:
                st.pool[st.hot_slot[l][e] * stride:(st.hot_slot[l][e] + 1) * stride].copy_(pinned)
            else:
                ld.host[e] = pinned
    torch.cuda.synchronize()
    return st, blobs


def run(st, mode, true_idx=None):
    outs = {}

    def grab(l, out):
        outs[l] = out.clone()

    stats = st.step(mode, true_idx=true_idx, on_layer=grab)
    torch.cuda.synchronize()
    return {l: o.cpu().numpy() for l, o in outs.items()}, stats


@pytest.mark.parametrize("n_stage", [4, 8])
def test_stack_modes_agree_and_match_oracle(mira, n_stage):
    cfg = SMALL_STACK
    st, blobs = build(mira, cfg, n_stage)
    true_idx = []
    for l in range(cfg.layers):
        mira.mira_moe_route(st.shape, st.args(l))
        torch.cuda.synchronize()
        true_idx.append(st.idx.cpu().numpy().copy())
    results = {}
    for mode in ("demand", "predict", "oracle"):
        st.reset_stage()
        for rep in range(2):  # the second step starts with slots left by the first
            outs, stats = run(st, mode, true_idx)
            results[mode, rep] = outs
            sel = sum(len(set(true_idx[l].reshape(-1).tolist())) for l in range(cfg.layers))
            assert stats.hot_hits + stats.stage_hits + stats.misses == sel
            if mode == "demand":  # slots may keep a layer's experts until the next step
                assert stats.prefetches == 0 and (rep > 0 or stats.stage_hits == 0)
            if mode == "oracle" and n_stage >= 8:
                # only layers 0 and 1 lack a lookahead
                cold01 = sum(len([e for e in set(true_idx[l].reshape(-1).tolist())
                                  if e not in st.hot_slot[l]]) for l in (0, 1))
                assert stats.misses <= cold01
    base = results["demand", 0]
    for key, outs in results.items():
        for l in range(cfg.layers):
            assert np.array_equal(outs[l], base[l]), (key, l)
    for l in range(cfg.layers):
        ld = st.layers[l]
        x = ld.x.float().cpu().numpy().astype(np.float64)
        wr = ld.w_router.float().cpu().numpy().astype(np.float64)
        b = None if ld.bias is None else ld.bias.cpu().numpy().astype(np.float64)
        ref = oracle.moe_forward(x, wr, b, [blobs[l, e] for e in range(cfg.E)], cfg.k, cfg.C, cfg.R)
        assert np.array_equal(ref["idx"], true_idx[l])
        assert_ffn_close(base[l], ref["out"], f"stack layer {l}")
