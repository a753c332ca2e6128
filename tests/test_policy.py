"""HOT-set telemetry and rebalancer (paper section IV-D): pure host logic."""
import pytest

from paper_2609_38090_amd.policy import RebalanceConfig, Rebalancer, Telemetry


def window(tel, traffic, tiers=None):
    """One window: traffic[e] tokens for expert e (served from tiers[e])."""
    for e, n in traffic.items():
        if n:
            tel.record(e, n, (tiers or {}).get(e, "hot"))
    tel.advance(sum(traffic.values()))


def test_telemetry_counts_tiers_and_windows():
    tel = Telemetry(4)
    window(tel, {0: 5, 1: 3, 2: 2}, {0: "hot", 1: "stage", 2: "cpu"})
    s = tel.stats
    assert (s[0].routed, s[0].hot, s[1].stage, s[2].cpu) == (5, 5, 3, 2)
    assert tel.tokens == 10 and s[2].last_use == 0
    tel.close_window()
    assert tel.tokens == 0 and s[0].routed == 0 and list(s[0].history) == [5]
    with pytest.raises(ValueError):
        tel.record(0, 1, "disk")


def test_cold_hot_expert_makes_way_after_probation():
    rb = Rebalancer(RebalanceConfig(interval=8, max_swaps=1, probation=2))
    tel = Telemetry(4)
    hot = {0, 1}
    # window 1: expert 3 bursts, expert 1 idle; 3 is still on probation
    window(tel, {0: 4, 3: 4}, {3: "cpu"})
    assert rb.due(tel)
    assert rb.plan(tel, hot) == []
    tel.close_window()
    # window 2: 3 again -> promoted in place of the idle expert 1
    window(tel, {0: 4, 3: 4}, {3: "cpu"})
    (sw,) = rb.plan(tel, hot)
    assert (sw.evict, sw.promote) == (1, 3)


def test_swaps_are_bounded_and_need_a_margin():
    cfg = RebalanceConfig(interval=1, max_swaps=2, probation=1, margin=1)
    rb = Rebalancer(cfg)
    tel = Telemetry(6)
    hot = {0, 1, 2}
    window(tel, {0: 3, 1: 1, 2: 2, 3: 9, 4: 8, 5: 2}, {3: "stage", 4: "cpu", 5: "cpu"})
    swaps = rb.plan(tel, hot)
    assert len(swaps) == 2                                   # bounded
    assert [(s.evict, s.promote) for s in swaps] == [(1, 4), (2, 3)]  # 4: 8 routed + 8 CPU-served
    # a candidate no better than the victim (plus margin) is not promoted
    tel2 = Telemetry(3)
    window(tel2, {0: 2, 1: 2}, {1: "stage"})
    assert Rebalancer(RebalanceConfig(interval=1, probation=1, miss_weight=0.0)).plan(tel2, {0}) == []


def test_victim_order_uses_recency_then_frequency():
    rb = Rebalancer(RebalanceConfig(interval=1, probation=1))
    tel = Telemetry(4)
    window(tel, {0: 1, 1: 1})     # clock 0
    tel.close_window()
    window(tel, {1: 0, 3: 5}, {3: "cpu"})  # 0 and 1 idle now; 1 used more recently? both last used at 0
    tel.stats[1].last_use = 1      # 1 was used later than 0
    (sw,) = rb.plan(tel, {0, 1})
    assert sw.evict == 0 and sw.promote == 3


def _random_telemetry(rng, n, windows):
    from paper_2609_38090_amd.policy import Telemetry
    tel = Telemetry(n)
    for w in range(windows):
        traffic = {e: int(rng.integers(0, 6)) if rng.random() < 0.6 else 0 for e in range(n)}
        tiers = {e: ["hot", "stage", "cpu"][int(rng.integers(0, 3))] for e in range(n)}
        for e, k in traffic.items():
            if k:
                tel.record(e, k, tiers[e])
        tel.advance(int(rng.integers(1, 9)))
        if w < windows - 1:
            tel.close_window()
    return tel


def test_native_planner_matches_the_reference_policy():
    """mira_rebalance_plan (the planner the native runtime runs) makes the same
    swaps as policy.Rebalancer.plan on random telemetry, settings and HOT sets."""
    import numpy as np
    import paper_2609_38090_amd as mira
    rng = np.random.default_rng(7)
    differ = 0
    for case in range(400):
        n = int(rng.integers(2, 17))
        cfg = RebalanceConfig(interval=8, max_swaps=int(rng.integers(0, 4)), probation=int(rng.integers(1, 4)),
                              miss_weight=float(rng.choice([0.0, 0.5, 1.0, 2.0])), margin=int(rng.integers(0, 3)))
        tel = _random_telemetry(rng, n, int(rng.integers(1, 12)))
        hot = set(int(e) for e in rng.choice(n, int(rng.integers(0, n + 1)), replace=False))
        want = [(s.evict, s.promote) for s in Rebalancer(cfg).plan(tel, hot)]
        hist = np.zeros((n, 8), np.int32)
        hl = np.zeros(n, np.int32)
        for e, st in enumerate(tel.stats):
            h = list(st.history)
            hist[e, :len(h)] = h
            hl[e] = len(h)
        c = mira.stack_config(1, 1, 0, 1, 256, rb_interval=cfg.interval, rb_max_swaps=cfg.max_swaps,
                              rb_probation=cfg.probation, rb_margin=cfg.margin, rb_miss_weight=cfg.miss_weight)
        got = mira.mira_rebalance_plan(c, [s.routed for s in tel.stats], [s.cpu for s in tel.stats],
                                       [s.last_use for s in tel.stats], hist, hl,
                                       [1 if e in hot else 0 for e in range(n)])
        assert got == want, (case, got, want)
        differ += bool(want)
    assert differ > 50  # enough cases actually swap
