"""Pins for the oracle's expert FFN, combine and predictor.

Expert weights are built on the quantization grid (w = q * sigma exactly), so
the packed format reproduces them exactly and the expected outputs can be
computed straight from the fp weights with torch (a library routine), without
going through the oracle's unpacking.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle


def _grid_weights(rng, C, R):
    """Grid weights: known int8 q and bf16 sigma; each row reaches |q| = 127 somewhere."""
    mant = rng.integers(128, 256, size=R).astype(np.float32)
    sigma = (mant * np.float32(2.0 ** -16)).astype(np.float32)
    qg = rng.integers(-100, 101, size=(R, C))
    qu = rng.integers(-100, 101, size=(R, C))
    qd = rng.integers(-100, 101, size=(C, R))
    qg[np.arange(R), rng.integers(0, C, size=R)] = 127
    wg = (qg * sigma[:, None]).astype(np.float32)
    wu = (qu * sigma[:, None]).astype(np.float32)
    wd = (qd * sigma[None, :]).astype(np.float32)
    return wg, wu, wd


def _torch_swiglu(x, wg, wu, wd):
    xt = torch.from_numpy(np.asarray(x, dtype=np.float64))
    g = xt @ torch.from_numpy(wg.astype(np.float64)).T
    u = xt @ torch.from_numpy(wu.astype(np.float64)).T
    return ((F.silu(g) * u) @ torch.from_numpy(wd.astype(np.float64)).T).numpy()


def test_single_expert_is_textbook_swiglu():
    rng = np.random.default_rng(0)
    C, R, T = 64, 128, 5
    wg, wu, wd = _grid_weights(rng, C, R)
    blob = oracle.pack_expert(wg, wu, wd)
    x = rng.standard_normal((T, C))
    y = oracle.expert_ffn(blob, x, C, R)
    ref = _torch_swiglu(x, wg, wu, wd)
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-15)
    # E = 1, k = 1 MoE layer reduces to the expert itself (weight 1)
    res = oracle.moe_forward(x, rng.standard_normal((1, C)), None, [blob], 1, C, R)
    assert np.allclose(res["out"], ref, rtol=1e-12, atol=1e-15)


def test_gate_and_up_roles_are_not_interchangeable():
    rng = np.random.default_rng(1)
    C, R = 64, 64
    wg, wu, wd = _grid_weights(rng, C, R)
    x = rng.standard_normal((3, C)) * 4
    y = oracle.expert_ffn(oracle.pack_expert(wg, wu, wd), x, C, R)
    swapped = _torch_swiglu(x, wu, wg, wd)
    assert not np.allclose(y, swapped, rtol=1e-3)


def test_zero_input_gives_zero_output():
    rng = np.random.default_rng(2)
    C, R, E = 64, 64, 4
    blobs = [oracle.pack_expert(*_grid_weights(rng, C, R)) for _ in range(E)]
    res = oracle.moe_forward(np.zeros((4, C)), rng.standard_normal((E, C)), rng.standard_normal(E),
                             blobs, 2, C, R)
    assert np.array_equal(res["out"], np.zeros((4, C)))


def test_dense_softmax_moe_when_k_equals_E():
    rng = np.random.default_rng(3)
    C, R, E, T = 64, 64, 4, 6
    ws = [_grid_weights(rng, C, R) for _ in range(E)]
    blobs = [oracle.pack_expert(*w) for w in ws]
    x = rng.standard_normal((T, C))
    wr = rng.standard_normal((E, C)) * 0.3
    b = rng.standard_normal(E)
    res = oracle.moe_forward(x, wr, b, blobs, E, C, R)
    probs = torch.softmax(torch.from_numpy(x @ wr.T + b), dim=1).numpy()
    ref = sum(probs[:, e:e + 1] * _torch_swiglu(x, *ws[e]) for e in range(E))
    assert np.allclose(res["out"], ref, rtol=1e-11, atol=1e-14)


def test_top2_weighted_combine_matches_closed_form():
    rng = np.random.default_rng(4)
    C, R, E, T = 64, 64, 6, 9
    ws = [_grid_weights(rng, C, R) for _ in range(E)]
    blobs = [oracle.pack_expert(*w) for w in ws]
    x = rng.standard_normal((T, C))
    wr = rng.standard_normal((E, C))
    res = oracle.moe_forward(x, wr, None, blobs, 2, C, R)
    lg = x @ wr.T
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-lg[t, e], e))[:2]
        w0 = 1.0 / (1.0 + np.exp(lg[t, order[1]] - lg[t, order[0]]))
        ref = w0 * _torch_swiglu(x[t:t + 1], *ws[order[0]]) + (1 - w0) * _torch_swiglu(x[t:t + 1], *ws[order[1]])
        assert np.allclose(res["out"][t], ref[0], rtol=1e-11, atol=1e-14)


def test_two_shared_experts_equal_one_double_width_expert():
    rng = np.random.default_rng(5)
    C, R, T = 64, 64, 7
    a = _grid_weights(rng, C, R)
    b = _grid_weights(rng, C, R)
    x = rng.standard_normal((T, C))
    ya = oracle.expert_ffn(oracle.pack_expert(*a), x, C, R)
    yb = oracle.expert_ffn(oracle.pack_expert(*b), x, C, R)
    cat = (np.concatenate([a[0], b[0]]), np.concatenate([a[1], b[1]]), np.concatenate([a[2], b[2]], axis=1))
    yab = oracle.expert_ffn(oracle.pack_expert(*cat), x, C, 2 * R)
    assert np.allclose(ya + yb, yab, rtol=1e-12, atol=1e-15)
    # shared experts enter the layer output with weight 1
    E = 2
    routed = [oracle.pack_expert(*_grid_weights(rng, C, R)) for _ in range(E)]
    wr = rng.standard_normal((E, C))
    base = oracle.moe_forward(x, wr, None, routed, 1, C, R)["out"]
    full = oracle.moe_forward(x, wr, None, routed, 1, C, R,
                              shared_blobs=[oracle.pack_expert(*a), oracle.pack_expert(*b)])["out"]
    assert np.allclose(full - base, yab, rtol=1e-10, atol=1e-13)


def test_relabelling_experts_leaves_output_unchanged():
    rng = np.random.default_rng(6)
    C, R, E, T, k = 64, 64, 5, 8, 2
    blobs = [oracle.pack_expert(*_grid_weights(rng, C, R)) for _ in range(E)]
    x = rng.standard_normal((T, C))
    wr = rng.standard_normal((E, C))
    b = rng.standard_normal(E)
    p = rng.permutation(E)
    out0 = oracle.moe_forward(x, wr, b, blobs, k, C, R)["out"]
    out1 = oracle.moe_forward(x, wr[p], b[p], [blobs[i] for i in p], k, C, R)["out"]
    assert np.allclose(out0, out1, rtol=1e-12, atol=1e-15)


def test_token_subset_matches_full_rows():
    rng = np.random.default_rng(7)
    C, R, E, T, k = 64, 64, 4, 10, 2
    blobs = [oracle.pack_expert(*_grid_weights(rng, C, R)) for _ in range(E)]
    x = rng.standard_normal((T, C))
    wr = rng.standard_normal((E, C))
    full = oracle.moe_forward(x, wr, None, blobs, k, C, R)["out"]
    sub = oracle.moe_forward(x, wr, None, blobs, k, C, R, tokens=[7, 2, 3])["out"]
    assert np.allclose(sub, full[[7, 2, 3]], rtol=1e-13, atol=1e-15)


def test_predictor_matches_torch_mlp():
    rng = np.random.default_rng(8)
    C, P, E, T, group = 48, 16, 8, 12, 4
    x = rng.standard_normal((T, C))
    w1 = rng.standard_normal((P, C)) / np.sqrt(C)
    b1 = rng.standard_normal(P) * 0.1
    w2 = rng.standard_normal((E, P)) / np.sqrt(P)
    b2 = rng.standard_normal(E) * 0.1
    s = oracle.predictor_scores(x, group, w1, b1, w2, b2)
    mlp = torch.nn.Sequential(torch.nn.Linear(C, P), torch.nn.ReLU(), torch.nn.Linear(P, E), torch.nn.Sigmoid()).double()
    with torch.no_grad():
        mlp[0].weight.copy_(torch.from_numpy(w1))
        mlp[0].bias.copy_(torch.from_numpy(b1))
        mlp[2].weight.copy_(torch.from_numpy(w2))
        mlp[2].bias.copy_(torch.from_numpy(b2))
        pooled = F.avg_pool1d(torch.from_numpy(x).T.unsqueeze(0), group).squeeze(0).T
        ref = mlp(pooled).numpy()
    assert np.allclose(s, ref, rtol=1e-12, atol=1e-15)
    with pytest.raises(ValueError):
        oracle.predictor_scores(x[:5], group, w1, b1, w2, b2)


def test_coverage_at_k():
    scores = np.array([0.1, 0.9, 0.5, 0.2])
    counts = np.array([10, 30, 40, 20])
    assert oracle.coverage_at_k(scores, counts, 1) == pytest.approx(0.3)
    assert oracle.coverage_at_k(scores, counts, 2) == pytest.approx(0.7)
    assert oracle.coverage_at_k(scores, counts, 4) == pytest.approx(1.0)
    assert oracle.coverage_at_k(scores, np.zeros(4), 2) == 0.0
