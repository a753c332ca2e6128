"""GPU parity of the MixtureHead predictor (section IV-E) against the oracle.

Tolerance, from the kernels' summation order (fp32, unit roundoff u = 2^-24;
weights are bf16, so exact in fp32): a sum whose every term passes through at
most K additions is off by at most K u times the sum of its terms' absolute
values (first order).  The pooled row passes `group` additions; a hidden unit
C/64 + 3 ceil(E/64) + 7 (a lane's sequential part, then a 64-lane tree); an
output logit ceil(P/64) + 7.  So with A, B, G the absolute-value sums of the
two heads' logits and the gate pre-activation (computed from |weights| and
|features|), and K the sum of the depths plus a margin,
  |dy| <= K u (A + B) + |da| |a - b|,  |da| <= K u G / 4 + 8u,
  |dp_e| <= p_e (2 max|dy| + 32u)     (softmax: d log p_e <= |dy_e| + max|dy|).
The top-m indicator and the histogram are integer decisions on exact counts,
so they agree exactly; a mismatch there shows up as a gross error.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from mira_inputs import MoEConfig, activations, mixture_weights, routing_sample

pytestmark = pytest.mark.gpu

U = 2.0 ** -24

# name, cid, C, E, k, m, Pa, Ph, N, group, T, act
CASES = [
    ("mix_small", 111, 256, 8, 2, 2, 64, 16, 8, 4, 12, "bf16"),        # 3 groups (< one chunk of 4)
    ("mix_ragged", 112, 192, 5, 2, 3, 70, 9, 6, 3, 27, "f32"),         # 9 groups: 2 chunks + 1, odd widths
    ("mix_beam", 113, 4096, 8, 2, 2, 512, 64, 8, 8, 8, "bf16"),        # one prediction per decode step
    ("mix_beam_all", 114, 4096, 8, 2, 2, 512, 64, 8, 8, 64, "bf16"),   # 8 steps batched
    ("mix_fine", 115, 2048, 64, 6, 6, 256, 128, 64, 16, 512, "bf16"),  # fine-grained source layer
    ("mix_wide", 116, 64, 256, 16, 16, 33, 200, 256, 2, 6, "f32"),     # E = N = 256, k = 16
    ("mix_group1", 117, 128, 4, 1, 1, 8, 8, 3, 1, 5, "bf16"),          # one token per prediction
]


def _run(mira, case):
    name, cid, C, E, k, m, Pa, Ph, N, group, T, act = case
    cfg = MoEConfig(name, cid, T=T, C=C, E=E, k=k, R=64, act=act, zipf_s=1.1)
    x = activations(cfg, 0, "cpu")
    logits, idx = routing_sample(cfg, 0)
    W = mixture_weights(cfg, 0, Pa, Ph, N)
    shape = mira.MixtureShape(C, E, k, m, Pa, Ph, N, group,
                              mira.MIRA_BF16 if act == "bf16" else mira.MIRA_F32)
    dev = {key: v.cuda() for key, v in W.items() if torch.is_tensor(v)}
    w = mira.MixtureWeights(**dev, bg=W["bg"])
    n = T // group
    ws = torch.empty(max(256, mira.mira_mixture_workspace_bytes(shape, T)), dtype=torch.uint8, device="cuda")
    probs = torch.full((n, N), float("nan"), dtype=torch.float32, device="cuda")
    alpha = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
    xd, ld, id_ = x.cuda(), logits.cuda(), idx.cuda()
    mira.mira_predict_mixture(shape, w, xd, ld, id_, T, probs, alpha, ws, ws.numel())
    torch.cuda.synchronize()
    W64 = {key: (v.double().numpy() if torch.is_tensor(v) else v) for key, v in W.items()}
    ref = oracle.mixture_head(x.double().numpy(), logits.double().numpy(), idx.numpy(), group, m, W64)
    return cfg, x, logits, idx, W64, ref, probs.cpu().double().numpy(), alpha.cpu().double().numpy()


def _bounds(case, x, logits, idx, W, ref):
    name, cid, C, E, k, m, Pa, Ph, N, group, T, act = case
    h, l, q, u = oracle.mixture_features(np.abs(x.double().numpy()), np.abs(logits.double().numpy()),
                                         idx.numpy(), group, E, m)
    A_ = {key: np.abs(v) if isinstance(v, np.ndarray) else abs(v) for key, v in W.items()}
    Sa = h @ A_["wah"].T + l @ A_["wal"].T + A_["ba1"]
    A = Sa @ A_["wa2"].T + A_["ba2"]
    Sh = q @ A_["whq"].T + u @ A_["whu"].T + A_["bh1"]
    B = Sh @ A_["wh2"].T + A_["bh2"]
    G = h @ A_["gh"] + l @ A_["gl"] + q @ A_["gq"] + u @ A_["gu"] + A_["bg"]
    K = group + C / 64 + 3 * math.ceil(E / 64) + math.ceil(max(Pa, Ph) / 64) + 32
    dalpha = K * U * G / 4 + 8 * U
    dy = K * U * (A + B) + dalpha[:, None] * np.abs(ref["a"] - ref["b"])
    return dalpha, dy


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_mixture_head_matches_oracle(mira, case):
    cfg, x, logits, idx, W, ref, probs, alpha = _run(mira, case)
    dalpha, dy = _bounds(case, x, logits, idx, W, ref)
    assert np.all(np.isfinite(probs)) and np.all(np.isfinite(alpha))
    assert np.all(np.abs(alpha - ref["alpha"]) <= dalpha), np.max(np.abs(alpha - ref["alpha"]) / dalpha)
    tol = ref["probs"] * (2 * dy.max(axis=1, keepdims=True) + 32 * U) + 1e-38
    err = np.abs(probs - ref["probs"])
    assert np.all(err <= tol), float(np.max(err / tol))
    assert np.allclose(probs.sum(axis=1), 1.0, atol=1e-5)


def test_mixture_head_histogram_branch_alone(mira):
    # Only the HistHead and the gate's indicator weights nonzero: the result is a
    # function of the exact integer features, and the top-m ties (experts 2 and
    # 4 with two pairs each) must resolve to the lower index as in the oracle.
    C, E, k, m, Pa, group = 64, 5, 2, 2, 1, 3
    Ph, N = 2 * E, E
    topk = torch.tensor([[1, 3], [3, 0], [1, 3], [4, 2], [2, 4], [0, 1]], dtype=torch.int32)
    Wn = {
        "wah": np.zeros((Pa, C)), "wal": np.zeros((Pa, E)), "ba1": np.zeros(Pa),
        "wa2": np.zeros((N, Pa)), "ba2": np.zeros(N),
        "whq": np.vstack([np.eye(E), np.zeros((E, E))]), "whu": np.vstack([np.zeros((E, E)), np.eye(E)]),
        "bh1": np.zeros(Ph), "wh2": np.hstack([np.eye(E), 3.0 * np.eye(E)]), "bh2": np.zeros(N),
        "gh": np.zeros(C), "gl": np.zeros(E), "gq": np.zeros(E), "gu": np.ones(E), "bg": -1.0,
    }
    shape = mira.MixtureShape(C, E, k, m, Pa, Ph, N, group, mira.MIRA_F32)
    dev = {key: torch.from_numpy(v).to(torch.bfloat16 if key[0] in "wg" else torch.float32).cuda()
           for key, v in Wn.items() if isinstance(v, np.ndarray)}
    w = mira.MixtureWeights(**dev, bg=Wn["bg"])
    x = torch.zeros((6, C), dtype=torch.float32)
    logits = torch.zeros((6, E), dtype=torch.float32)
    ws = torch.empty(mira.mira_mixture_workspace_bytes(shape, 6), dtype=torch.uint8, device="cuda")
    probs = torch.empty((2, N), dtype=torch.float32, device="cuda")
    alpha = torch.empty((2,), dtype=torch.float32, device="cuda")
    mira.mira_predict_mixture(shape, w, x.cuda(), logits.cuda(), topk.cuda(), 6, probs, alpha, ws, ws.numel())
    torch.cuda.synchronize()
    ref = oracle.mixture_head(x.numpy(), logits.numpy(), topk.numpy(), group, m, Wn)
    # two flagged experts per group: alpha = sigmoid(2 - 1)
    assert np.allclose(alpha.cpu().numpy(), 1.0 / (1.0 + math.exp(-1.0)), rtol=1e-6)
    assert np.allclose(probs.cpu().numpy(), ref["probs"], rtol=1e-5, atol=1e-7)
    assert np.array_equal(np.argsort(-probs.cpu().numpy(), axis=1, kind="stable")[:, :2],
                          np.argsort(-ref["probs"], axis=1, kind="stable")[:, :2])



def test_mixture_head_groups_are_independent(mira):
    """A group's prediction does not depend on the other groups of the call:
    1 and 4 groups (features built inside the hidden layer's kernel) and 5
    groups (separate features kernel) give the same bits for the groups they
    share, and match the oracle."""
    name, cid, C, E, k, m, Pa, Ph, N, group, T, act = CASES[2]  # the beam shape
    cfg = MoEConfig(name, cid, T=40, C=C, E=E, k=k, R=64, act=act, zipf_s=1.1)
    x = activations(cfg, 0, "cpu")
    logits, idx = routing_sample(cfg, 0)
    W = mixture_weights(cfg, 0, Pa, Ph, N)
    shape = mira.MixtureShape(C, E, k, m, Pa, Ph, N, group, mira.MIRA_BF16)
    w = mira.MixtureWeights(**{key: v.cuda() for key, v in W.items() if torch.is_tensor(v)}, bg=W["bg"])
    xd, ld, id_ = x.cuda(), logits.cuda(), idx.cuda()
    out = {}
    for t in (40, 32, 8):
        n = t // group
        ws = torch.full((max(256, mira.mira_mixture_workspace_bytes(shape, t)),), 0xFF, dtype=torch.uint8,
                        device="cuda")
        probs = torch.empty((n, N), dtype=torch.float32, device="cuda")
        alpha = torch.empty((n,), dtype=torch.float32, device="cuda")
        mira.mira_predict_mixture(shape, w, xd[:t], ld[:t], id_[:t], t, probs, alpha, ws, ws.numel())
        torch.cuda.synchronize()
        out[t] = (probs.cpu().numpy(), alpha.cpu().numpy())
    for t in (32, 8):
        n = t // group
        assert np.array_equal(out[t][0], out[40][0][:n]), t
        assert np.array_equal(out[t][1], out[40][1][:n]), t
    W64 = {key: (v.double().numpy() if torch.is_tensor(v) else v) for key, v in W.items()}
    ref = oracle.mixture_head(x.double().numpy(), logits.double().numpy(), idx.numpy(), group, m, W64)
    assert np.allclose(out[40][0], ref["probs"], rtol=1e-4, atol=1e-7)
