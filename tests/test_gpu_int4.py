"""GPU parity of the INT4 variant (MIRA_FLAG_INT4: 4-bit values, fp16 scale per
row and 64-column group) against the oracle.

Bars: the device packer's bytes equal the oracle's; routing as in the INT8
path (bit-exact); the layer output within the same rel-Frobenius 5e-3 and
max-abs 2e-2 * rms(out) bars, and in practice within decode_rel_floor (the
int8 matrix-core sums are exact per group; the rounding is the fixed-point
step of the activations and the fp32 group scaling)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_layer import EPS, Layer, decode_rel_floor, run_and_check
from mira_inputs import CONFIGS, MoEConfig

pytestmark = pytest.mark.gpu

# the INT4 layout needs hidden and ffn multiples of 128
SMALL_BF16 = MoEConfig("i4_bf16", 121, T=16, C=128, E=8, k=2, R=256, zipf_s=1.2)
SMALL_FG = MoEConfig("i4_fg", 122, T=16, C=128, E=64, k=6, R=128, S=2, zipf_s=1.0)
SMALL_F32 = MoEConfig("i4_f32", 123, T=16, C=128, E=3, k=3, R=128, act="f32")
WIDE = MoEConfig("i4_wide", 124, T=16, C=4096, E=4, k=2, R=384, zipf_s=0.5)   # C at the LDS-digit limit
TALL = MoEConfig("i4_tall", 125, T=16, C=4224, E=4, k=2, R=256, zipf_s=0.5)   # past it: digits from L2


def test_device_pack_int4_bit_exact(mira):
    lay = Layer(CONFIGS["tiny"], fmt="int4")
    for e in range(4):
        ref = oracle.pack_expert_int4(*lay.master(e), eps=EPS)
        assert np.array_equal(lay.slot_bytes(int(lay.table[e])), ref), e


def test_device_pack_int4_bf16_input_and_padding(mira):
    C, R, n = 128, 256, 3
    g = torch.Generator().manual_seed(6)
    w = [torch.randn((n, *s), generator=g).mul_(sc).to(torch.bfloat16)
         for s, sc in (((R, C), 0.03), ((R, C), 1e-6), ((C, R), 2.0))]
    stride = mira.mira_packed_expert_bytes_int4(C, R) + 512
    out = torch.full((n * stride,), 0x5A, dtype=torch.uint8, device="cuda")
    mira.mira_pack_experts(mira.MoEShape(C, R, 1, 1, flags=mira.MIRA_FLAG_INT4), n, mira.MIRA_BF16,
                           *(t.cuda() for t in w), EPS, out, stride, 1)
    got = out.cpu().numpy().reshape(n, stride)
    for e in range(n):
        ref = oracle.pack_expert_int4(*(t[e].float().numpy() for t in w), eps=EPS)
        assert np.array_equal(got[e, :ref.size], ref), e
        assert not got[e, ref.size:].any()


@pytest.mark.parametrize("cfg,T", [(CONFIGS["tiny"], 16), (SMALL_BF16, 1), (SMALL_BF16, 3), (SMALL_BF16, 5),
                                   (SMALL_BF16, 8), (SMALL_BF16, 16), (SMALL_FG, 1), (SMALL_FG, 2),
                                   (SMALL_FG, 16),
                                   (SMALL_F32, 5), (SMALL_F32, 11), (WIDE, 1), (WIDE, 4), (WIDE, 9),
                                   (TALL, 2), (TALL, 7)])
def test_int4_decode_matches_oracle(mira, cfg, T):
    lay = Layer(cfg, T=T, fmt="int4")
    res, errs, _, _ = run_and_check(lay)
    assert errs[0] < decode_rel_floor(T), errs   # far inside the bar


def test_int4_two_phase_and_repeat_bit_identical(mira):
    lay = Layer(SMALL_BF16, T=7, fmt="int4")
    a = lay.run()
    b = lay.run(two_phase=True)
    c = lay.run()
    for key in a:
        assert np.array_equal(a[key], b[key]), key
        assert np.array_equal(a[key], c[key]), key


def test_int4_non_resident_expert_sets_status(mira):
    # the LDS-digit gate/up kernel returns before its barrier for a missing
    # expert; the other experts' outputs are still written
    lay = Layer(SMALL_BF16, T=5, fmt="int4", resident=[1, 2, 3, 4, 5, 6, 7])
    res = lay.run()
    assert res["counts"][0] > 0 and res["status"][0] & 1
    assert np.all(np.isfinite(res["out"]))
    lay2 = Layer(SMALL_BF16, T=1, fmt="int4")
    lay2.table[int(lay2.run()["idx"][0, 0])] = 99   # beyond n_slots: skipped, flagged
    assert lay2.run()["status"][0] & 2


def test_int4_rejects_prefill(mira):
    lay = Layer(SMALL_BF16, T=4, fmt="int4")
    with pytest.raises(mira.MiraError) as ei:
        lay.run(mira.MIRA_FLAG_FORCE_PREFILL)
    assert ei.value.code == -6


@pytest.mark.slow
def test_int4_mixtral_decode_layer(mira):
    lay = Layer(CONFIGS["mixtral_decode"], fmt="int4")
    res, errs, blobs, ties = run_and_check(lay)
    for e, ref in blobs.cache.items():
        assert np.array_equal(lay.slot_bytes(int(lay.table[e])), ref), f"expert {e} bytes differ"
    assert len(blobs.cache) == 2
    print(f"mixtral decode int4: rel_fro={errs[0]:.2e} max_abs/rms={errs[1]:.2e}")
