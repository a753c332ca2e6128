"""One-token calls on the GPU against the oracle.  A one-token call splits
the 16-row tiles of all active experts evenly over the CUs (W waves per
workgroup, W = ceil(tiles / CUs) up to 8), gives every tile of H' its own
exponent, and the down kernel one operand column per (tile, digit) pair;
the gate/up kernel hands the slot it resolved to the down kernel.  These
shapes cover tile counts far below one per CU, a ragged last workgroup, the
8-wave cap with more workgroups than CUs, one active expert, shared
experts, more than 64 experts (the general preparation path), fp32
activations, both weight formats, and the INT4 fallback to the block kernel
above C = 4096.  Bars: routing bit-exact and every output
row within the error bars (run_and_check), and the decode floor of one
token."""
import numpy as np
import pytest

import oracle
from gpu_layer import Layer, LazyBlobs, assert_ffn_close, check_routing, decode_rel_floor, run_and_check
from mira_inputs import MoEConfig

pytestmark = pytest.mark.gpu


def _cfg(name, cid, **kw):
    return MoEConfig(name, cid, T=1, **kw)


CASES = [
    # 2 active experts x 8 tiles = 16 tiles: one wave per workgroup
    ("few_tiles", _cfg("one_few", 601, C=256, E=4, k=2, R=128), "int8"),
    # a shared expert beside the routed ones: 3 x 64 tiles
    ("shared", _cfg("one_shared", 602, C=512, E=8, k=2, R=1024, S=1, zipf_s=1.0), "int8"),
    # the fine-grained shape: 8 active x 88 tiles = 704 -> 3 waves, the last
    # workgroup two tiles short
    ("fine_grained", _cfg("one_fg", 603, C=2048, E=64, k=6, R=1408, S=2, zipf_s=1.0), "int8"),
    # 10 active x 256 tiles = 2560 -> the 8-wave cap, 320 workgroups
    ("wave_cap", _cfg("one_cap", 604, C=256, E=16, k=8, R=4096, S=2), "int8"),
    # one active expert
    ("one_expert", _cfg("one_e1", 605, C=384, E=1, k=1, R=640), "int8"),
    # fp32 activations
    ("f32", _cfg("one_f32", 606, C=384, E=5, k=3, R=640, act="f32"), "int8"),
    ("int4_few_tiles", _cfg("one_i4_few", 607, C=256, E=4, k=2, R=128), "int4"),
    ("int4_shared", _cfg("one_i4_shared", 608, C=1024, E=8, k=2, R=1536, S=1, zipf_s=1.2), "int4"),
    # C above the LDS staging limit: the INT4 block kernel without staging
    ("int4_wide", _cfg("one_i4_wide", 609, C=4224, E=4, k=2, R=256), "int4"),
    # more than 64 experts: the general preparation path (two experts per
    # lane in the top-k) in front of the tile kernels
    ("many_experts", _cfg("one_e96", 611, C=256, E=96, k=4, R=128, S=1, zipf_s=1.0), "int8"),
    ("int4_many_experts", _cfg("one_i4_e96", 612, C=256, E=96, k=4, R=128, S=1, zipf_s=1.0), "int4"),
]


@pytest.mark.parametrize("cfg,fmt", [pytest.param(c, f, id=i) for i, c, f in CASES])
def test_one_token_shapes(mira, cfg, fmt):
    tiles = min(cfg.G, cfg.k + cfg.S) * (cfg.R // 16)
    assert tiles > 0
    res, errs, _, _ = run_and_check(Layer(cfg, fmt=fmt))
    assert errs[0] < decode_rel_floor(1), (errs, tiles)


@pytest.mark.parametrize("fmt", ["int8", "int4"])
def test_one_token_missing_selected_expert(mira, fmt):
    """The token's first selected expert is not resident: the gate/up kernel
    flags it (status bit 0) and stores -1 as its slot, the down kernel skips
    it, and out holds every other term.  The workspace starts as NaN bytes,
    so a read of the missing expert's never-written H' would show."""
    cfg = _cfg("one_missing", 610, C=512, E=8, k=2, R=768, zipf_s=1.0)
    probe = Layer(cfg, fmt=fmt).run()
    e0 = int(probe["idx"][0][0])
    lay = Layer(cfg, fmt=fmt, resident=[e for e in range(cfg.E) if e != e0])
    res = lay.run(ws_fill=0xFF)
    assert res["status"][0] == 1
    o_x, o_wr, o_b = lay.oracle_inputs()
    o_logits = oracle.router_logits(o_x, o_wr, o_b)
    assert not check_routing(res, lay, o_logits)
    assert int(res["idx"][0][0]) == e0

    class _Zero:
        def __init__(self, blobs):
            self.blobs = blobs

        def __len__(self):
            return len(self.blobs)

        def __getitem__(self, e):
            if e == e0:  # not resident: the bytes of an expert with zero weights and scales
                return np.zeros_like(self.blobs[(e0 + 1) % cfg.E])
            return self.blobs[e]

    ref = oracle.moe_forward(o_x, o_wr, o_b, _Zero(LazyBlobs(lay)), cfg.k, cfg.C, cfg.R, fmt=fmt)["out"]
    assert np.isfinite(res["out"]).all()
    assert_ffn_close(res["out"], ref, f"one token, expert {e0} missing, {fmt}")


@pytest.mark.parametrize("fmt", ["int8", "int4"])
def test_one_token_reads_nothing_stale_from_the_workspace(mira, fmt):
    """Every tile exponent, digit and resolved slot the down kernel reads is
    written in the same call: a workspace filled with NaN bytes and one filled
    with zero bytes give bit-identical outputs.  (A one-token call right
    after a 16-token call on the same scratch is the no-alloc test's case.)"""
    cfg = _cfg("one_ws", 613, C=512, E=8, k=2, R=1024, S=1, zipf_s=1.0)
    lay = Layer(cfg, fmt=fmt)
    a = lay.run(ws_fill=0xFF)
    b = lay.run(ws_fill=0x00)
    for key in ("out", "idx", "w", "counts", "status"):
        assert np.array_equal(a[key], b[key]), key
    assert np.isfinite(a["out"]).all()
