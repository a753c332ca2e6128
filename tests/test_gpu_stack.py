"""A stack of MoE layers over HOT and STAGE slots (paper sections IV-C, IV-E,
IV-F): every layer's output must be the same whether an expert is served from
its HOT slot, a STAGE slot filled ahead of time or a demand copy, and must
match the oracle (each layer on its own seeded input)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_layer import EPS, assert_ffn_close
from mira_inputs import (MoEConfig, activations, expert_weights, mixture_weights, predictor_weights,
                         resident_experts, router_bias, router_weights)

pytestmark = pytest.mark.gpu

MIX_PA, MIX_PH = 48, 16  # MixtureHead widths of the small stack

SMALL_STACK = MoEConfig("small_stack", 104, T=8, C=128, E=8, k=2, R=192, zipf_s=1.2, layers=5, resident=4,
                        pred_hidden=32, pred_group=8)
# the INT4 layout needs hidden and ffn multiples of 128
SMALL_STACK_I4 = MoEConfig("small_stack_i4", 105, T=8, C=128, E=8, k=2, R=256, zipf_s=1.2, layers=5,
                           resident=4, pred_hidden=32, pred_group=8)


def _head(mira, cfg, l, head):
    if l + 2 >= cfg.layers:
        return None
    if head == "mlp":
        return tuple(t.cuda() for t in predictor_weights(cfg, l, "cpu"))
    W = mixture_weights(cfg, l, MIX_PA, MIX_PH)
    return mira.MixtureWeights(**{k: v.cuda() for k, v in W.items() if torch.is_tensor(v)}, bg=W["bg"])


def build(mira, cfg, n_stage, hot=None, bias=None, host_all=False, rebalancer=None, head="mlp",
          fmt="int8", vram_mode="large", **stack_kw):
    from paper_2609_38090_amd.stack import ExpertStack, LayerData
    i4 = fmt == "int4"
    flag = mira.MIRA_FLAG_INT4 if i4 else 0
    stride = (mira.mira_packed_expert_bytes_int4 if i4 else mira.mira_packed_expert_bytes)(cfg.C, cfg.R)
    layers, blobs = [], {}
    for l in range(cfg.layers):
        b = router_bias(cfg, l) if bias is None else bias(l)
        pred = _head(mira, cfg, l, head)
        layers.append(LayerData(x=activations(cfg, l, "cuda"), w_router=router_weights(cfg, l, "cuda"),
                                bias=None if b is None else b.cuda(),
                                hot=resident_experts(cfg, l) if hot is None else hot(l), pred=pred))
    shape = mira.MoEShape(cfg.C, cfg.R, cfg.E, cfg.k, cfg.S, mira.MIRA_BF16, flag)
    ps = (mira.PredShape(cfg.C, cfg.pred_hidden, cfg.E, cfg.pred_group, mira.MIRA_BF16) if head == "mlp" else
          mira.MixtureShape(cfg.C, cfg.E, cfg.k, cfg.k, MIX_PA, MIX_PH, cfg.E, cfg.pred_group, mira.MIRA_BF16))
    st = ExpertStack(shape, cfg.T, layers, stride, n_stage=n_stage, pred_shape=ps, rebalancer=rebalancer,
                     vram_mode=vram_mode, **stack_kw)
    pack_shape = mira.MoEShape(cfg.C, cfg.R, 1, 1, flags=flag)
    hot_slot = st.hot_slot
    for l, ld in enumerate(layers):
        for e in range(cfg.E):
            w = [np.ascontiguousarray(t.numpy()) for t in expert_weights(cfg, l, e, "cpu")]
            # the oracle's own packing, for the reference
            blobs[l, e] = (oracle.pack_expert_int4 if i4 else oracle.pack_expert)(*w, eps=EPS)
            pinned = torch.zeros(stride, dtype=torch.uint8).pin_memory()
            mira.mira_pack_experts(pack_shape, 1, mira.MIRA_F32, w[0].ctypes.data, w[1].ctypes.data,
                                   w[2].ctypes.data, EPS, pinned, stride, 0)
            if e in hot_slot[l]:
                st.pool[hot_slot[l][e] * stride:(hot_slot[l][e] + 1) * stride].copy_(pinned)
            if host_all or e not in hot_slot[l]:
                ld.host[e] = pinned
    torch.cuda.synchronize()
    return st, blobs


def oracle_layer(st, cfg, blobs, l, fmt="int8"):
    """The oracle's output of layer l of the stack on the layer's current input and bias."""
    ld = st.layers[l]
    x = ld.x.float().cpu().numpy().astype(np.float64)
    wr = ld.w_router.float().cpu().numpy().astype(np.float64)
    b = None if ld.bias is None else ld.bias.cpu().numpy().astype(np.float64)
    return oracle.moe_forward(x, wr, b, [blobs[l, e] for e in range(cfg.E)], cfg.k, cfg.C, cfg.R, fmt=fmt)


def true_routing(mira, st, cfg):
    out = []
    for l in range(cfg.layers):
        mira.mira_moe_route(st.shape, st.args(l))
        torch.cuda.synchronize()
        out.append(st.idx.cpu().numpy().copy())
    return out


def run(st, mode, true_idx=None):
    outs = {}

    def grab(l, out):
        outs[l] = out.clone()

    stats = st.step(mode, true_idx=true_idx, on_layer=grab)
    torch.cuda.synchronize()
    return {l: o.cpu().numpy() for l, o in outs.items()}, stats


@pytest.mark.parametrize("n_stage,fmt", [(4, "int8"), (8, "int8"), (4, "int4")])
def test_stack_modes_agree_and_match_oracle(mira, n_stage, fmt):
    cfg = SMALL_STACK if fmt == "int8" else SMALL_STACK_I4
    st, blobs = build(mira, cfg, n_stage, fmt=fmt)
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
        ref = oracle.moe_forward(x, wr, b, [blobs[l, e] for e in range(cfg.E)], cfg.k, cfg.C, cfg.R, fmt=fmt)
        assert np.array_equal(ref["idx"], true_idx[l])
        assert_ffn_close(base[l], ref["out"], f"stack layer {l}")


def test_rebalancer_tracks_drift_without_changing_outputs(mira):
    """Expert popularity moves at step 6; the rebalanced stack must swap the
    new popular experts into HOT (telemetry, probation, bounded swaps) while
    every layer output stays bit-identical to the stack whose HOT set is fixed."""
    from paper_2609_38090_amd.policy import RebalanceConfig, Rebalancer
    from mira_inputs import drift_bias, drift_hot
    cfg = SMALL_STACK
    hot0 = lambda l: drift_hot(cfg, l, 0, cfg.resident)  # noqa: E731
    b0 = lambda l: drift_bias(cfg, l, 0)  # noqa: E731
    fixed, _ = build(mira, cfg, 4, hot=hot0, bias=b0, host_all=True)
    moving, blobs = build(mira, cfg, 4, hot=hot0, bias=b0, host_all=True,
                          rebalancer=Rebalancer(RebalanceConfig(interval=32, max_swaps=1, probation=2)))
    swaps = 0
    kinds = set()
    log = []
    for s in range(24):
        ep = s // 6
        for st in (fixed, moving):
            for l, ld in enumerate(st.layers):
                ld.x.copy_(activations(cfg, l, "cuda", base=1 + s))
                ld.bias.copy_(drift_bias(cfg, l, ep).cuda())
        a, _ = run(fixed, "demand")
        b, stats = run(moving, "demand" if s % 2 else "predict")
        swaps += stats.swaps
        evs = moving.events()
        log += evs
        kinds |= {ev[0] for ev in evs}
        for l in range(cfg.layers):
            assert np.array_equal(a[l], b[l]), (s, l)
        if s in (11, 23):  # after swaps: the rebalanced stack against the oracle
            for l in range(cfg.layers):
                assert_ffn_close(b[l], oracle_layer(moving, cfg, blobs, l)["out"], f"step {s} layer {l}")
    assert swaps > 0
    assert "evict" in kinds and kinds & {"swap_relabel", "swap_copy"}
    # the rebalanced HOT sets hold more of the last period's popular experts
    last = [set(drift_hot(cfg, l, 3, cfg.resident)) for l in range(cfg.layers)]
    got_fixed = sum(len(fixed.hot_set(l) & last[l]) for l in range(cfg.layers))
    got_moving = sum(len(moving.hot_set(l) & last[l]) for l in range(cfg.layers))
    assert got_moving > got_fixed, (got_moving, got_fixed)
    # HOT is a role that relabelling moves between slots: mira_stack_set_hot
    # takes exactly the slots that are HOT now, whatever their index
    hot_now = {slot: (l, e) for l in range(cfg.layers) for e, slot in moving.hot_slot[l].items()}
    assert any(ev[0] == "swap_relabel" for ev in log)
    assert len(hot_now) == moving.n_hot and set(hot_now) != set(range(moving.n_hot))
    for slot in range(moving.n_slots):
        if slot in hot_now:
            mira.mira_stack_set_hot(moving.handle, *hot_now[slot], slot, copy=False)
        else:
            with pytest.raises(mira.MiraError):
                mira.mira_stack_set_hot(moving.handle, 0, 0, slot, copy=False)


def test_stack_with_mixture_head_stages_its_top_experts(mira):
    """Predictive staging driven by the MixtureHead: outputs stay bit-identical
    to demand fetching, and the experts requested for layer l+2 are the two with
    the largest MixtureHead probability summed over the step's groups (oracle
    on the layer's routing record; checked where the ranking has a clear gap)."""
    cfg = SMALL_STACK
    st, _ = build(mira, cfg, 8, head="mixture")
    dem, _ = run(st, "demand")
    st.reset_stage()
    st.events()  # drop the earlier steps' log
    routing = {}

    def grab(l, out):
        routing[l] = (st.logits.cpu().numpy().copy(), st.idx.cpu().numpy().copy(), out.clone())

    stats = st.step("predict", on_layer=grab)
    torch.cuda.synchronize()
    log = st.events()
    requested = [(t, e) for (kind, l, t, e, slot) in log if kind == "predicted"]
    for l in range(cfg.layers):
        assert np.array_equal(routing[l][2].cpu().numpy(), dem[l]), l
    assert stats.prefetches + stats.prefetch_cached + stats.prefetch_declined == 2 * (cfg.layers - 2)
    checked = 0
    for l in range(cfg.layers - 2):
        W = mixture_weights(cfg, l, MIX_PA, MIX_PH)
        W64 = {k: (v.double().numpy() if torch.is_tensor(v) else v) for k, v in W.items()}
        x = st.layers[l].x.float().cpu().numpy().astype(np.float64)
        logits, idx, _ = routing[l]
        ref = oracle.mixture_head(x, logits.astype(np.float64), idx, cfg.pred_group, cfg.k, W64)["probs"].sum(0)
        order = np.argsort(-ref, kind="stable")
        if ref[order[1]] - ref[order[2]] < 1e-4:
            continue
        want = set(order[:2].tolist())
        got = {e for (t, e) in requested if t == l + 2}
        assert got == want, (l, got, want)
        # every pick was staged, found cached, or declined
        fate = {e: kind for (kind, ll, t, e, slot) in log if t == l + 2 and ll == l and
                kind in ("prefetch", "prefetch_cached", "prefetch_declined")}
        assert set(fate) == want
        for e in want & st.hot_set(l + 2):
            assert fate[e] == "prefetch_cached"
        checked += 1
    assert checked > 0


def test_small_vram_mode_frees_stage_slots_after_their_layer(mira):
    """Small-VRAM mode (section IV-C): a STAGE slot is released right after its
    layer, so no slot holds an expert once the step is over and a second step
    finds nothing staged; outputs equal the large-VRAM stack's and the oracle's."""
    cfg = SMALL_STACK
    small, blobs = build(mira, cfg, 4, vram_mode="small")
    large, _ = build(mira, cfg, 4)
    true_idx = true_routing(mira, small, cfg)
    for mode in ("oracle", "demand", "predict"):
        for rep in range(2):
            a, sa = run(small, mode, true_idx)
            b, sb = run(large, mode, true_idx)
            for l in range(cfg.layers):
                assert np.array_equal(a[l], b[l]), (mode, rep, l)
            assert all(small.staged(l, e) < 0 for l in range(cfg.layers) for e in range(cfg.E))
            if mode == "demand":
                assert sa.stage_hits == 0
    for l in range(cfg.layers):
        assert_ffn_close(a[l], oracle_layer(small, cfg, blobs, l)["out"], f"small layer {l}")


def test_stage_capacity_zero_with_every_expert_hot(mira):
    """No STAGE slot at all: with every expert HOT nothing is ever copied, each
    prediction is a skipped ("cached") prefetch, and outputs match the oracle."""
    cfg = SMALL_STACK
    st, blobs = build(mira, cfg, 0, hot=lambda l: list(range(cfg.E)))
    st.events()
    outs, stats = run(st, "predict")
    log = st.events()
    assert stats.misses == 0 and stats.stage_hits == 0 and stats.h2d_bytes == 0
    assert stats.prefetches == 0 and stats.prefetch_declined == 0
    assert stats.prefetch_cached == 2 * (cfg.layers - 2)
    assert {k for (k, *_ ) in log} <= {"hot_hit", "predicted", "prefetch_cached"}
    for l in range(cfg.layers):
        assert_ffn_close(outs[l], oracle_layer(st, cfg, blobs, l)["out"], f"layer {l}")


def test_stage_capacity_one_declines_and_drops_prefetches(mira):
    """One STAGE slot beside 7 of 8 experts HOT per layer.  The non-HOT
    expert of layers 0 and 1 is one they do not select, that of layers 2, 3
    and 4 one they do.  In oracle mode, layer 0 prefetches layer 2's expert
    into the slot; at layer 1 the slot still holds that prefetch for the next
    layer, so the prefetch for layer 3 is declined; layer 2 hits its staged
    expert; later demand copies may take a prefetch for a later layer (it is
    dropped).  Outputs equal demand fetching and the oracle."""
    cfg = SMALL_STACK
    probe, _ = build(mira, cfg, 0, hot=lambda l: list(range(cfg.E)))
    sel = [set(r.reshape(-1).tolist()) for r in true_routing(mira, probe, cfg)]
    del probe
    if any(len(sel[l]) == cfg.E for l in (0, 1)):
        pytest.skip("layers 0 and 1 select every expert at this seed")
    cold = [min(set(range(cfg.E)) - sel[l]) if l < 2 else min(sel[l]) for l in range(cfg.layers)]
    st, blobs = build(mira, cfg, 1, hot=lambda l: [e for e in range(cfg.E) if e != cold[l]], host_all=True)
    true_idx = true_routing(mira, st, cfg)
    dem, _ = run(st, "demand")
    st.reset_stage()
    st.events()
    outs, stats = run(st, "oracle", true_idx)
    log = st.events()
    assert ("prefetch", 0, 2, cold[2], st.n_hot) in log
    assert ("prefetch_declined", 1, 3, cold[3], -1) in log
    assert ("stage_hit", 2, 2, cold[2], st.n_hot) in log
    assert stats.prefetch_declined >= 1 and stats.stage_hits >= 1
    for rep in range(2):
        for l in range(cfg.layers):
            assert np.array_equal(outs[l], dem[l]), (rep, l)
        outs, _ = run(st, "oracle", true_idx)
    for l in range(cfg.layers):
        assert_ffn_close(dem[l], oracle_layer(st, cfg, blobs, l)["out"], f"layer {l}")


def test_coverage_of_the_mlp_head_matches_the_oracle(mira):
    """Coverage@m (section VI-B, mass-weighted): the runtime counts, for each
    layer l+2 it predicted, the routed pairs landing on the head's m picks.
    Its totals equal the sum over the picks it logged, and on every layer
    whose oracle top-m ranking has a clear gap the picks are the oracle head's
    and the covered mass is the oracle's coverage_at_k against the true
    routing."""
    cfg = SMALL_STACK
    st, blobs = build(mira, cfg, 8)
    true_idx = true_routing(mira, st, cfg)
    st.events()
    _, stats = run(st, "predict")
    log = st.events()
    m = st.stage_per_layer
    num = tot = checked = 0
    for l in range(cfg.layers - 2):
        counts = np.bincount(true_idx[l + 2].reshape(-1), minlength=cfg.E)
        picks = [e for (k, ll, t, e, slot) in log if k == "predicted" and t == l + 2]
        assert len(picks) == m
        num += int(counts[picks].sum())
        tot += int(counts.sum())
        w1, b1, w2, b2 = (t.float().cpu().numpy() for t in st.layers[l].pred)
        x = st.layers[l].x.float().cpu().numpy().astype(np.float64)
        sc = oracle.predictor_scores(x, cfg.pred_group, w1, b1, w2, b2).sum(axis=0)
        srt = np.sort(sc)[::-1]
        if srt[m - 1] - srt[m] < 1e-5:
            continue
        assert set(picks) == set(np.argsort(-sc, kind="stable")[:m].tolist()), l
        assert int(counts[picks].sum()) == round(oracle.coverage_at_k(sc, counts, m) * counts.sum()), l
        checked += 1
    assert (stats.cov_hits, stats.cov_total) == (num, tot)
    assert checked > 0
    print(f"Coverage@{m} of the untrained MLP head: {stats.coverage:.3f} ({checked} layers checked)")
