"""Pins for the oracle's router, top-k, combine weights and permutation (section II-A)."""
import numpy as np
import pytest
import torch

import oracle


def test_router_logits_one_hot_rows_pick_columns():
    rng = np.random.default_rng(0)
    C, E = 16, 5
    wg = rng.standard_normal((E, C))
    b = rng.standard_normal(E)
    x = np.zeros((3, C))
    x[0, 4] = 1.0
    x[1, 0] = 2.0
    x[2, 15] = -1.0
    lg = oracle.router_logits(x, wg, b)
    assert np.allclose(lg[0], wg[:, 4] + b, rtol=0, atol=1e-15)
    assert np.allclose(lg[1], 2 * wg[:, 0] + b, rtol=0, atol=1e-15)
    assert np.allclose(lg[2], -wg[:, 15] + b, rtol=0, atol=1e-15)
    assert np.array_equal(oracle.router_logits(np.zeros((2, C)), wg, None), np.zeros((2, E)))


@pytest.mark.parametrize("E,k", [(4, 2), (8, 2), (8, 8), (64, 6), (5, 1)])
def test_topk_matches_exhaustive_sort(E, k):
    rng = np.random.default_rng(E * 10 + k)
    # small integers make exact ties common
    lg = rng.integers(-3, 4, size=(200, E)).astype(np.float64)
    idx = oracle.topk_select(lg, k)
    for t in range(lg.shape[0]):
        brute = sorted(range(E), key=lambda e: (-lg[t, e], e))[:k]
        assert idx[t].tolist() == brute


def test_topk_rejects_nonfinite_and_bad_k():
    with pytest.raises(ValueError):
        oracle.topk_select(np.array([[0.0, np.nan]]), 1)
    with pytest.raises(ValueError):
        oracle.topk_select(np.zeros((1, 3)), 4)


def test_near_tie_detection():
    lg = np.array([[1.0, 0.99995, -1.0, -2.0],     # top-2 within delta
                   [1.0, 0.5, 0.49999, 0.0],      # 2nd vs 3rd (the k+1-th) within delta
                   [1.0, 0.5, 0.0, -0.5]])
    assert oracle.near_tie_tokens(lg, 2, 1e-4).tolist() == [0, 1]


def test_combine_weights_closed_forms():
    rng = np.random.default_rng(5)
    lg = rng.standard_normal((50, 8))
    idx = oracle.topk_select(lg, 2)
    w = oracle.combine_weights(lg, idx)
    l0 = lg[np.arange(50), idx[:, 0]]
    l1 = lg[np.arange(50), idx[:, 1]]
    assert np.allclose(w[:, 0], 1.0 / (1.0 + np.exp(l1 - l0)), rtol=1e-14, atol=0)
    assert np.allclose(w.sum(1), 1.0, rtol=0, atol=1e-15)
    w1 = oracle.combine_weights(lg, oracle.topk_select(lg, 1))
    assert np.all(w1 == 1.0)
    # equal selected logits share the weight evenly
    flat = np.zeros((1, 6))
    assert np.allclose(oracle.combine_weights(flat, oracle.topk_select(flat, 3)), 1.0 / 3)
    # without renormalisation: the selected entries of the full softmax
    wf = oracle.combine_weights(lg, idx, norm_topk=False)
    sm = torch.softmax(torch.from_numpy(lg), dim=1).numpy()
    assert np.allclose(wf, np.take_along_axis(sm, idx.astype(np.int64), 1), rtol=1e-13, atol=0)


@pytest.mark.parametrize("T,E,k,S", [(16, 4, 2, 0), (37, 8, 2, 0), (50, 64, 6, 2), (1, 8, 2, 0), (0, 4, 2, 1)])
def test_permutation_properties(T, E, k, S):
    rng = np.random.default_rng(T + E)
    lg = rng.standard_normal((T, E))
    idx = oracle.topk_select(lg, k) if T else np.zeros((0, k), dtype=np.int32)
    counts, offsets, perm, inv = oracle.permute_pairs(idx, E, S)
    P = T * k + S * T
    group = np.concatenate([idx.reshape(-1), np.repeat(np.arange(E, E + S), T)]).astype(np.int64)
    # counts are the histogram; offsets its exclusive scan
    assert np.array_equal(counts, np.bincount(group, minlength=E + S))
    assert offsets[0] == 0 and offsets[-1] == P and np.all(np.diff(offsets) == counts)
    # bijection
    assert sorted(perm.tolist()) == list(range(P))
    assert np.array_equal(perm[inv], np.arange(P))
    # equal to a brute-force stable sort by (group, pair index)
    assert perm.tolist() == sorted(range(P), key=lambda p: (group[p], p))
    for g in range(E + S):
        seg = perm[offsets[g]:offsets[g + 1]]
        assert np.all(group[seg] == g)
        assert np.all(np.diff(seg) > 0)
