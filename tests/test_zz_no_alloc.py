"""GPU check of the workspace-free layer call (mira_moe_forward_noalloc)
against the call with a caller workspace (mira_moe_forward): the outputs of
two calls in a row, the second with fewer tokens (so the scratch still holds
the first call's contents), equal the workspace call's bit for bit."""
import numpy as np
import pytest
import torch

import paper_2609_38090_amd as mira
from gpu_layer import Layer
from mira_inputs import CONFIGS, MoEConfig

pytestmark = pytest.mark.gpu

MEDIUM = MoEConfig("noalloc_medium", 109, T=64, C=512, E=8, k=2, R=1024, zipf_s=1.2)


def _call(lay, T, noalloc, flags=0):
    c = lay.cfg
    s = lay.shape(flags)
    dev = lay.device
    P = T * c.k + c.S * T
    r = dict(out=torch.full((T, c.C), float("nan"), dtype=torch.float32, device=dev),
             idx=torch.full((T, c.k), -7, dtype=torch.int32, device=dev),
             w=torch.zeros((T, c.k), dtype=torch.float32, device=dev),
             logits=torch.zeros((T, c.E), dtype=torch.float32, device=dev),
             counts=torch.zeros((c.G,), dtype=torch.int32, device=dev),
             status=torch.full((1,), -1, dtype=torch.int32, device=dev),
             offsets=torch.zeros((c.G + 1,), dtype=torch.int32, device=dev),
             order=torch.full((max(P, 1),), -1, dtype=torch.int32, device=dev))
    ws = None if noalloc else torch.empty(mira.mira_workspace_bytes(s, T), dtype=torch.uint8, device=dev)
    a = mira.MoEArgs(x=lay.x[:T], n_tokens=T, n_slots=lay.n_slots, w_router=lay.wr, router_bias=lay.bias,
                     slot_table=lay.table, slot_pool=lay.pool, slot_stride=lay.stride, out=r["out"],
                     topk_idx=r["idx"], topk_weight=r["w"], logits=r["logits"], expert_counts=r["counts"],
                     status=r["status"], expert_offsets=r["offsets"], pair_order=r["order"],
                     workspace=ws, workspace_bytes=0 if ws is None else ws.numel())
    (mira.mira_moe_forward_noalloc if noalloc else mira.mira_moe_forward)(s, a)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in r.items()}


def _same(a, b, what):
    for key in a:
        assert np.array_equal(a[key], b[key]), f"{what}: {key}"
    assert a["status"][0] == 0


@pytest.mark.parametrize("cfg,T1,T2", [(MEDIUM, 64, 5), (CONFIGS["mixtral_decode"], 16, 1)],
                         ids=["medium_prefill_then_decode", "mixtral_decode_16_then_1"])
def test_noalloc_matches_workspace_call_twice(mira, cfg, T1, T2):
    print(f"[noalloc {cfg.name} T={T1} then T={T2}]", flush=True)
    lay = Layer(cfg, T=T1)
    for T in (T1, T2):
        got = _call(lay, T, noalloc=True)
        ref = _call(lay, T, noalloc=False)
        _same(got, ref, f"{cfg.name} T={T}")
    # and again in the other order of the two kinds of call, now forced onto
    # the prefill kernels at the smaller size
    got = _call(lay, T2, noalloc=True, flags=mira.MIRA_FLAG_FORCE_PREFILL)
    ref = _call(lay, T2, noalloc=False, flags=mira.MIRA_FLAG_FORCE_PREFILL)
    _same(got, ref, f"{cfg.name} T={T2} prefill")


def test_noalloc_rejects_a_call_beyond_the_scratch(mira):
    lay = Layer(MEDIUM, T=1)
    s = lay.shape()
    T = next(t for t in range(64, 1 << 16, 64)
             if mira.mira_workspace_bytes(s, t) > mira.MIRA_NOALLOC_SCRATCH_BYTES)
    a = mira.MoEArgs(x=lay.x, n_tokens=T, n_slots=lay.n_slots, w_router=lay.wr, slot_table=lay.table,
                     slot_pool=lay.pool, slot_stride=lay.stride, out=lay.x)
    with pytest.raises(mira.MiraError) as e:
        mira.mira_moe_forward_noalloc(s, a)
    assert e.value.code == -4
