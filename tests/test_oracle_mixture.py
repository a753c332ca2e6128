"""Pins for the oracle's MixtureHead (section IV-E).

Each case fixes a value by hand or by a closed form, chosen so that a dropped
term, a transposed weight, a wrong gate direction or mixing probabilities
instead of logits fails at least one of them.
"""
import math

import numpy as np
import pytest

import oracle


def _zero_weights(C, E, Pa, Ph, N):
    return {
        "wah": np.zeros((Pa, C)), "wal": np.zeros((Pa, E)), "ba1": None,
        "wa2": np.zeros((N, Pa)), "ba2": None,
        "whq": np.zeros((Ph, E)), "whu": np.zeros((Ph, E)), "bh1": None,
        "wh2": np.zeros((N, Ph)), "bh2": None,
        "gh": np.zeros(C), "gl": np.zeros(E), "gq": np.zeros(E), "gu": np.zeros(E), "bg": 0.0,
    }


def _routing():
    # 2 groups of 3 tokens, k = 2, E = 5
    topk = np.array([[1, 3], [3, 0], [1, 3],      # group 0: counts 0:1 1:2 3:3
                     [4, 2], [2, 4], [0, 1]])     # group 1: counts 0:1 1:1 2:2 4:2
    return topk


def test_features_by_hand():
    C, E, group, m = 4, 5, 3, 2
    x = np.arange(6 * C, dtype=np.float64).reshape(6, C)
    logits = np.arange(6 * E, dtype=np.float64).reshape(6, E) * 0.5
    h, l, q, u = oracle.mixture_features(x, logits, _routing(), group, E, m)
    assert np.array_equal(h[0], x[:3].mean(axis=0)) and np.array_equal(h[0], [4, 5, 6, 7])
    assert np.array_equal(l[1], [10.0, 10.5, 11.0, 11.5, 12.0])
    assert np.array_equal(q[0], np.array([1, 2, 0, 3, 0]) / 6.0)
    assert np.array_equal(q[1], np.array([1, 1, 2, 0, 2]) / 6.0)
    # top-2: group 0 -> experts 3 (3 pairs) and 1 (2); group 1 -> 2 and 4 tie at 2
    assert np.array_equal(u[0], [0, 1, 0, 1, 0])
    assert np.array_equal(u[1], [0, 0, 1, 0, 1])


def test_top_m_ties_prefer_lower_index_and_skip_empty_experts():
    E = 6
    topk = np.array([[5, 2], [4, 1]])  # one group of 2 tokens: four experts with one pair each
    x, logits = np.zeros((2, 64)), np.zeros((2, E))
    _, _, _, u = oracle.mixture_features(x, logits, topk, 2, E, 3)
    assert np.array_equal(u[0], [0, 1, 1, 0, 1, 0])
    _, _, _, u = oracle.mixture_features(x, logits, topk, 2, E, 6)  # m beyond the used experts
    assert np.array_equal(u[0], [0, 1, 1, 0, 1, 1])


def test_zero_head_is_uniform_with_half_gate():
    C, E, Pa, Ph, N = 8, 5, 3, 4, 7
    rng = np.random.default_rng(0)
    r = oracle.mixture_head(rng.standard_normal((6, C)), rng.standard_normal((6, E)), _routing(), 3, 2,
                            _zero_weights(C, E, Pa, Ph, N))
    assert np.array_equal(r["alpha"], [0.5, 0.5])
    assert np.allclose(r["probs"], 1.0 / N, rtol=0, atol=1e-15)


def test_heads_mix_logits_not_probabilities():
    # alpha = 1/2, a = (2, 0), b = (0, 0): mixed logits (1, 0) -> p0 = e / (e + 1).
    # Mixing the two distributions instead would give 0.5 * e^2/(e^2+1) + 0.25.
    C, E, Pa, Ph, N = 4, 5, 2, 2, 2
    W = _zero_weights(C, E, Pa, Ph, N)
    W["ba2"] = np.array([2.0, 0.0])
    r = oracle.mixture_head(np.zeros((6, C)), np.zeros((6, E)), _routing(), 3, 2, W)
    assert r["probs"][0, 0] == pytest.approx(math.e / (math.e + 1), rel=1e-15)
    assert np.array_equal(r["y"][0], [1.0, 0.0])


def test_gate_weights_each_feature():
    C, E, Pa, Ph, N = 4, 5, 1, 1, 3
    rng = np.random.default_rng(1)
    x = rng.standard_normal((6, C))
    logits = rng.standard_normal((6, E))
    sig = lambda v: 1.0 / (1.0 + math.exp(-v))  # noqa: E731
    for name, expect in (("gh", lambda i: x[3 * i:3 * i + 3, 2].mean()),
                         ("gl", lambda i: logits[3 * i:3 * i + 3, 2].mean()),
                         ("gq", lambda i: [0.0, 2 / 6.0][i]),      # expert 2: 0 pairs, then 2
                         ("gu", lambda i: [0.0, 1.0][i])):         # expert 2 in the top-2 of group 1 only
        W = _zero_weights(C, E, Pa, Ph, N)
        W[name] = np.zeros(C if name == "gh" else E)
        W[name][2] = 1.0
        W["bg"] = 0.25
        r = oracle.mixture_head(x, logits, _routing(), 3, 2, W)
        for i in range(2):
            assert r["alpha"][i] == pytest.approx(sig(expect(i) + 0.25), rel=1e-14), name


def test_gate_direction_selects_acthead():
    # alpha -> weight of the ActHead: with alpha = sigmoid(3) the ActHead's logits carry
    # weight sigmoid(3), the HistHead's 1 - sigmoid(3).
    C, E, Pa, Ph, N = 4, 5, 1, 1, 2
    W = _zero_weights(C, E, Pa, Ph, N)
    W["ba2"] = np.array([1.0, 0.0])
    W["bh2"] = np.array([0.0, 1.0])
    W["bg"] = 3.0
    r = oracle.mixture_head(np.zeros((6, C)), np.zeros((6, E)), _routing(), 3, 2, W)
    s = 1.0 / (1.0 + math.exp(-3.0))
    assert np.allclose(r["y"][0], [s, 1 - s], rtol=1e-15)


def test_acthead_permutation_weights_pick_pooled_columns():
    # wah = a permutation P (not symmetric), wa2 = I: a = ReLU(P h).  A transposed
    # weight would apply P^-1 and pick other columns.
    C, E, N = 4, 5, 4
    perm = [2, 0, 3, 1]
    W = _zero_weights(C, E, C, 1, N)
    W["wah"] = np.eye(C)[perm]
    W["wa2"] = np.eye(N)
    x = np.array([[1.0, -2.0, 3.0, 4.0], [3.0, 2.0, -1.0, 0.0], [2.0, 3.0, 1.0, 2.0]] * 2)
    h = x[:3].mean(axis=0)  # (2, 1, 1, 2)
    r = oracle.mixture_head(x, np.zeros((6, E)), _routing(), 3, 2, W)
    assert np.array_equal(r["a"][0], np.maximum(h[perm], 0.0))
    # ReLU: a negative pooled column contributes nothing
    x2 = -x
    r = oracle.mixture_head(x2, np.zeros((6, E)), _routing(), 3, 2, W)
    assert np.array_equal(r["a"][0], np.zeros(N))


def test_acthead_router_logit_part_and_biases():
    C, E, N = 4, 5, 5
    W = _zero_weights(C, E, E, 1, N)
    W["wal"] = np.eye(E)[[4, 3, 2, 1, 0]]
    W["wa2"] = np.eye(N)
    W["ba1"] = np.full(E, 10.0)   # keeps ReLU open
    W["ba2"] = np.arange(N, dtype=np.float64)
    logits = np.arange(30, dtype=np.float64).reshape(6, E)
    r = oracle.mixture_head(np.zeros((6, C)), logits, _routing(), 3, 2, W)
    lbar = logits[:3].mean(axis=0)
    assert np.array_equal(r["a"][0], lbar[::-1] + 10.0 + np.arange(N))


def test_histhead_histogram_and_indicator_parts():
    C, E, N = 4, 5, 5
    W = _zero_weights(C, E, 1, 2 * E, N)
    W["whq"] = np.vstack([np.eye(E), np.zeros((E, E))])
    W["whu"] = np.vstack([np.zeros((E, E)), np.eye(E)])
    W["wh2"] = np.hstack([np.eye(E), 10.0 * np.eye(E)])
    W["bh2"] = np.full(N, -1.0)
    r = oracle.mixture_head(np.zeros((6, C)), np.zeros((6, E)), _routing(), 3, 2, W)
    assert np.allclose(r["b"][0], np.array([1, 2, 0, 3, 0]) / 6.0 + 10.0 * np.array([0, 1, 0, 1, 0]) - 1.0,
                       rtol=1e-15, atol=0)
    assert np.allclose(r["b"][1], np.array([1, 1, 2, 0, 2]) / 6.0 + 10.0 * np.array([0, 0, 1, 0, 1]) - 1.0,
                       rtol=1e-15, atol=0)


def test_softmax_shift_and_output_permutation():
    rng = np.random.default_rng(2)
    C, E, Pa, Ph, N = 16, 5, 6, 4, 7
    W = {
        "wah": rng.standard_normal((Pa, C)), "wal": rng.standard_normal((Pa, E)), "ba1": rng.standard_normal(Pa),
        "wa2": rng.standard_normal((N, Pa)), "ba2": rng.standard_normal(N),
        "whq": rng.standard_normal((Ph, E)), "whu": rng.standard_normal((Ph, E)), "bh1": rng.standard_normal(Ph),
        "wh2": rng.standard_normal((N, Ph)), "bh2": rng.standard_normal(N),
        "gh": rng.standard_normal(C), "gl": rng.standard_normal(E), "gq": rng.standard_normal(E),
        "gu": rng.standard_normal(E), "bg": 0.1,
    }
    x, logits = rng.standard_normal((6, C)), rng.standard_normal((6, E))
    r = oracle.mixture_head(x, logits, _routing(), 3, 2, W)
    assert np.allclose(r["probs"].sum(axis=1), 1.0, rtol=0, atol=1e-15)
    W2 = dict(W, ba2=W["ba2"] + 5.0, bh2=W["bh2"] + 5.0)   # alpha + (1 - alpha) = 1
    assert np.allclose(oracle.mixture_head(x, logits, _routing(), 3, 2, W2)["probs"], r["probs"],
                       rtol=1e-13, atol=1e-16)
    p = rng.permutation(N)
    W3 = dict(W, wa2=W["wa2"][p], ba2=W["ba2"][p], wh2=W["wh2"][p], bh2=W["bh2"][p])
    assert np.allclose(oracle.mixture_head(x, logits, _routing(), 3, 2, W3)["probs"], r["probs"][:, p],
                       rtol=1e-14, atol=1e-17)


def test_rejects_bad_arguments():
    x, logits = np.zeros((6, 4)), np.zeros((6, 5))
    with pytest.raises(ValueError):
        oracle.mixture_features(x[:5], logits[:5], _routing()[:5], 3, 5, 2)
    with pytest.raises(ValueError):
        oracle.mixture_features(x, logits, _routing(), 3, 5, 0)
    with pytest.raises(ValueError):
        oracle.mixture_features(x, logits, _routing() + 1, 3, 5, 2)
