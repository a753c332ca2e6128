"""CPU checks of the C ABI: the library loads, exports every declared entry
point, rejects bad arguments before any launch, and its host packer is
byte-exact against the oracle (paper section IV-B)."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import oracle
import paper_2609_38090_amd as mira
from mira_inputs import CONFIGS, expert_weights

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "mira.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mira_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    lib = mira.load()
    declared = _declared_functions()
    assert len(declared) >= 14
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(mira.EXPORTED_SYMBOLS) == declared
    assert "gfx950" in mira.mira_version()


def test_packed_expert_bytes_closed_form():
    for C, R in [(256, 512), (4096, 14336), (2048, 1408), (64, 64), (8, 1)]:
        assert mira.mira_packed_expert_bytes(C, R) == oracle.packed_expert_bytes(C, R)
    assert mira.mira_packed_expert_bytes(0, 64) == 0
    assert mira.mira_packed_expert_bytes(64, -1) == 0


@pytest.mark.parametrize("shape", [(2048, 1408, 64, 6, 2), (4096, 14336, 8, 2, 0), (64, 8192, 256, 16, 0),
                                   (256, 4096, 16, 8, 2), (128, 64, 1, 1, 0)])
def test_workspace_bytes_monotone_and_validated(shape):
    # a workspace sized for max_tokens must serve every smaller call, also a
    # one-token call, whose H' exponents are per 16-row tile instead of per
    # 64-row block
    s = mira.MoEShape(*shape, mira.MIRA_BF16)
    sizes = [mira.mira_workspace_bytes(s, t) for t in list(range(1, 40)) + [512, 2048]]
    assert all(a <= b for a, b in zip(sizes, sizes[1:]))
    assert all(v % 256 == 0 for v in sizes)
    with pytest.raises(mira.MiraError):
        mira.mira_workspace_bytes(mira.MoEShape(100, 1408, 64, 6), 4)   # hidden not a multiple of 64


@pytest.mark.parametrize("bad,code", [
    (dict(hidden=100), -2), (dict(ffn=0), -2), (dict(top_k=9), -2), (dict(top_k=0), -2),
    (dict(n_experts=250, n_shared=10), -2), (dict(act_dtype=7), -1), (dict(flags=0x100), -1),
    (dict(flags=mira.MIRA_FLAG_FORCE_DECODE | mira.MIRA_FLAG_FORCE_PREFILL), -1),
])
def test_forward_rejects_bad_shapes_before_launch(bad, code):
    kw = dict(hidden=256, ffn=512, n_experts=8, top_k=2, n_shared=0, act_dtype=mira.MIRA_F32, flags=0)
    kw.update(bad)
    a = mira.MoEArgs(n_tokens=4)
    with pytest.raises(mira.MiraError) as ei:
        mira.mira_moe_forward(mira.MoEShape(**kw), a, stream=1)
    assert ei.value.code == code
    assert mira.mira_last_error()


def test_forward_argument_checks():
    s = mira.MoEShape(256, 512, 4, 2, 0, mira.MIRA_F32)
    ws = mira.mira_workspace_bytes(s, 16)
    base = dict(x=0x1000, n_tokens=16, n_slots=4, w_router=0x2000, slot_table=0x3000, slot_pool=0x10000,
                slot_stride=oracle.packed_expert_bytes(256, 512), out=0x4000, workspace=0x20000,
                workspace_bytes=ws)
    cases = [
        (dict(x=None), -1), (dict(n_slots=0), -1), (dict(x=0x1004), -3), (dict(slot_pool=0x10010), -3),
        (dict(slot_stride=256), -2), (dict(workspace_bytes=ws - 256), -4), (dict(n_tokens=-1), -2),
        (dict(workspace=0x20040), -3),
    ]
    for change, code in cases:
        kw = dict(base)
        kw.update(change)
        with pytest.raises(mira.MiraError) as ei:
            mira.mira_moe_forward(s, mira.MoEArgs(**kw), stream=1)
        assert ei.value.code == code, (change, mira.mira_last_error())
    s2 = mira.MoEShape(256, 512, 4, 2, 0, mira.MIRA_F32, mira.MIRA_FLAG_FORCE_DECODE)
    kw = dict(base, n_tokens=17, workspace_bytes=10**12)
    with pytest.raises(mira.MiraError) as ei:
        mira.mira_moe_forward(s2, mira.MoEArgs(**kw), stream=1)
    assert ei.value.code == -2
    # zero tokens is a no-op that touches nothing
    mira.mira_moe_forward(s, mira.MoEArgs(n_tokens=0), stream=1)


def test_predict_and_stage_argument_checks():
    p = mira.PredShape(4096, 512, 8, 8)
    assert mira.mira_predict_workspace_bytes(p, 16) >= 2 * 4096 * 4
    with pytest.raises(mira.MiraError):
        mira.mira_predict(p, 0x1000, 12, 0x2000, None, 0x3000, None, 0x4000, 0x5000, 10**9, stream=1)
    with pytest.raises(mira.MiraError):
        mira.mira_stage_expert(0x1000, 256, 0, 0x2000, 512, copy_stream=1)
    with pytest.raises(mira.MiraError):
        mira.mira_set_slot(0x1000, 0, -2, stream=1)


def _host_pack(C, R, wg, wu, wd, eps=1e-8, dtype=mira.MIRA_F32, stride=None):
    n = wg.shape[0]
    stride = stride or oracle.packed_expert_bytes(C, R)
    out = np.full((n, stride), 0xAB, dtype=np.uint8)
    mira.mira_pack_experts(mira.MoEShape(C, R, 1, 1), n, dtype, wg.ctypes.data, wu.ctypes.data,
                           wd.ctypes.data, eps, out.ctypes.data, stride, 0)
    return out


def test_host_pack_matches_oracle_tiny_config():
    cfg = CONFIGS["tiny"]
    ws = [expert_weights(cfg, 0, e) for e in range(cfg.E)]
    wg = np.stack([w[0].numpy() for w in ws])
    wu = np.stack([w[1].numpy() for w in ws])
    wd = np.stack([w[2].numpy() for w in ws])
    got = _host_pack(cfg.C, cfg.R, wg, wu, wd)
    for e in range(cfg.E):
        assert np.array_equal(got[e], oracle.pack_expert(wg[e], wu[e], wd[e]))


def test_host_pack_bf16_input_and_padded_stride():
    rng = np.random.default_rng(0)
    C, R = 128, 192
    w = [torch.from_numpy(rng.standard_normal((2, *s)).astype(np.float32) * 0.05).to(torch.bfloat16)
         for s in ((R, C), (R, C), (C, R))]
    bits = [t.view(torch.int16).numpy().view(np.uint16).copy() for t in w]
    stride = oracle.packed_expert_bytes(C, R) + 512
    got = _host_pack(C, R, *bits, dtype=mira.MIRA_BF16, stride=stride)
    for e in range(2):
        ref = oracle.pack_expert(*(t[e].float().numpy() for t in w))
        assert np.array_equal(got[e, :ref.size], ref)
        assert not got[e, ref.size:].any()


def test_host_pack_fine_grained_expert_slice():
    """One expert of the fine-grained layer at full size (C=2048, R=1408)."""
    cfg = CONFIGS["fine_grained"]
    wg, wu, wd = (t.numpy()[None] for t in expert_weights(cfg, 0, 5))
    got = _host_pack(cfg.C, cfg.R, wg, wu, wd)
    assert np.array_equal(got[0], oracle.pack_expert(wg[0], wu[0], wd[0]))


def test_mixture_head_argument_checks():
    shape = dict(hidden=64, n_src=4, top_k=2, hist_top=2, act_hidden=8, hist_hidden=8, n_out=4, group=2,
                 act_dtype=mira.MIRA_F32)
    good = mira.MixtureShape(**shape)
    ws = mira.mira_mixture_workspace_bytes(good, 4)
    assert ws > 0 and ws % 256 == 0
    assert mira.mira_mixture_workspace_bytes(good, 8) >= ws
    w = mira.MixtureWeights(**{n: 0x1000 * (i + 1) for i, n in enumerate(
        ("wah", "wal", "ba1", "wa2", "ba2", "whq", "whu", "bh1", "wh2", "bh2", "gh", "gl", "gq", "gu"))})
    args = dict(x=0x100000, logits=0x200000, topk_idx=0x300000, n_tokens=4, probs=0x400000, alpha=None,
                workspace=0x500000, workspace_bytes=ws)
    mira.mira_predict_mixture(good, w, **dict(args, n_tokens=0), stream=1)   # no-op
    for change, code in [(dict(hidden=100), -2), (dict(n_src=0), -2), (dict(n_src=257), -2),
                         (dict(top_k=17), -2), (dict(hist_top=5), -2), (dict(hist_top=0), -2),
                         (dict(act_hidden=0), -2), (dict(n_out=300), -2), (dict(group=0), -2),
                         (dict(act_dtype=5), -1)]:
        with pytest.raises(mira.MiraError) as ei:
            mira.mira_predict_mixture(mira.MixtureShape(**dict(shape, **change)), w, **args, stream=1)
        assert ei.value.code == code, change
    for change, code in [(dict(n_tokens=3), -2), (dict(x=None), -1), (dict(x=0x100008), -3),
                         (dict(workspace=0x500010), -3), (dict(workspace_bytes=ws - 256), -4)]:
        with pytest.raises(mira.MiraError) as ei:
            mira.mira_predict_mixture(good, w, **dict(args, **change), stream=1)
        assert ei.value.code == code, change
    for field, val in (("gq", None), ("wah", 0x1008)):
        bad = mira.MixtureWeights(**{**w.__dict__, field: val})
        with pytest.raises(mira.MiraError):
            mira.mira_predict_mixture(good, bad, **args, stream=1)


def _host_pack_i4(C, R, wg, wu, wd, dtype=mira.MIRA_F32, eps=1e-8, stride=None):
    n = wg.shape[0]
    stride = stride or oracle.packed_expert_bytes_int4(C, R)
    out = np.full((n, stride), 0xAB, dtype=np.uint8)
    mira.mira_pack_experts(mira.MoEShape(C, R, 1, 1, flags=mira.MIRA_FLAG_INT4), n, dtype, wg.ctypes.data,
                           wu.ctypes.data, wd.ctypes.data, eps, out.ctypes.data, stride, 0)
    return out


def test_int4_packed_bytes_match_oracle():
    for C, R in [(4096, 14336), (2048, 1408), (128, 128), (256, 512)]:
        assert mira.mira_packed_expert_bytes_int4(C, R) == oracle.packed_expert_bytes_int4(C, R)
    assert mira.mira_packed_expert_bytes_int4(0, 128) == 0
    assert mira.mira_packed_expert_bytes_int4(64, 128) == 0     # the INT4 layout needs multiples of 128


def test_host_pack_int4_matches_oracle():
    """Random weights at three magnitudes (the smallest gives fp16 subnormal
    scales), planted ties, all-zero and overflowing groups; fp32 and bf16."""
    rng = np.random.default_rng(11)
    C, R = 128, 256
    w = [rng.standard_normal((3, *s)).astype(np.float32) for s in ((R, C), (R, C), (C, R))]
    for t, scale in zip(w, (0.05, 1e-6, 3.0)):
        t *= scale
    w[0][0, 3, :64] = 0.0                       # an all-zero group
    w[1][1, 5, 64:128] = 0.0
    w[1][1, 5, 70] = 7e5                        # the scale saturates at 65504
    w[0][2, 0, :6] = [7.0 * (1 + 2 ** -11), 3.5, 0.5, 1.5, 2.5, -3.5]   # ties
    w[0][2, 0, 6:64] = 0.0
    stride = oracle.packed_expert_bytes_int4(C, R) + 256
    got = _host_pack_i4(C, R, *w, stride=stride)
    for e in range(3):
        ref = oracle.pack_expert_int4(w[0][e], w[1][e], w[2][e])
        assert np.array_equal(got[e, :ref.size], ref), e
        assert not got[e, ref.size:].any()
    wb = [torch.from_numpy(t).to(torch.bfloat16) for t in w]
    bits = [t.view(torch.int16).numpy().view(np.uint16).copy() for t in wb]
    got = _host_pack_i4(C, R, *bits, dtype=mira.MIRA_BF16)
    for e in range(3):
        assert np.array_equal(got[e], oracle.pack_expert_int4(*(t[e].float().numpy() for t in wb))), e


def test_int4_forward_argument_checks():
    C, R = 256, 512
    s = mira.MoEShape(C, R, 4, 2, 0, mira.MIRA_F32, flags=mira.MIRA_FLAG_INT4)
    ws = mira.mira_workspace_bytes(s, 16)
    base = dict(x=0x1000, n_tokens=4, n_slots=4, w_router=0x2000, slot_table=0x3000, slot_pool=0x10000,
                slot_stride=oracle.packed_expert_bytes_int4(C, R), out=0x4000, workspace=0x20000,
                workspace_bytes=ws)
    for shape_flags, change, code in [
            (mira.MIRA_FLAG_INT4 | mira.MIRA_FLAG_FORCE_PREFILL, {}, -6),
            (mira.MIRA_FLAG_INT4, dict(n_tokens=17), -6),
            (mira.MIRA_FLAG_INT4, dict(slot_stride=oracle.packed_expert_bytes_int4(C, R) - 256), -2)]:
        sh = mira.MoEShape(C, R, 4, 2, 0, mira.MIRA_F32, flags=shape_flags)
        with pytest.raises(mira.MiraError) as ei:
            mira.mira_moe_forward(sh, mira.MoEArgs(**dict(base, **change)), stream=1)
        assert ei.value.code == code, (shape_flags, change)
    for hidden, ffn in [(192, 512), (256, 448)]:   # INT4 needs multiples of 128
        sh = mira.MoEShape(hidden, ffn, 4, 2, 0, mira.MIRA_F32, flags=mira.MIRA_FLAG_INT4)
        with pytest.raises(mira.MiraError) as ei:
            mira.mira_moe_forward(sh, mira.MoEArgs(**base), stream=1)
        assert ei.value.code == -2
        with pytest.raises(mira.MiraError):
            _host_pack_i4(hidden, ffn, *(np.zeros((1, *sh_), dtype=np.float32)
                                         for sh_ in ((ffn, hidden), (ffn, hidden), (hidden, ffn))),
                          stride=256 * 1024)


def test_host_pack_int4_matches_header_formulas():
    """The library's host packer, read back through the header's INT4 offset
    formulas (not through the oracle), stores the intended integers and
    scales."""
    import int4_layout as hl
    C, R = 256, 128
    (wg, wu, wd), q, sc = hl.marked_weights(C, R)
    stride = mira.mira_packed_expert_bytes_int4(C, R)
    out = np.zeros(stride, dtype=np.uint8)
    mira.mira_pack_experts(mira.MoEShape(C, R, 1, 1, flags=mira.MIRA_FLAG_INT4), 1, mira.MIRA_F32,
                           wg.ctypes.data, wu.ctypes.data, wd.ctypes.data, 1e-8, out.ctypes.data, stride, 0)
    for (gq, gs), name in zip(hl.decode_blob(out, C, R), ("gate", "up", "down")):
        assert np.array_equal(gq, q[name]), name
        assert np.array_equal(gs.astype(np.float64), sc[name]), name


def test_noalloc_forward_argument_checks():
    """The workspace-free call rejects a caller workspace and a call that would
    not fit the library's scratch, before touching the GPU."""
    C, R = 4096, 14336
    s = mira.MoEShape(C, R, 8, 2, 0, mira.MIRA_BF16)
    a = mira.MoEArgs(x=0x1000, n_tokens=1, n_slots=8, w_router=0x2000, slot_table=0x3000,
                     slot_pool=0x10000, slot_stride=mira.mira_packed_expert_bytes(C, R), out=0x4000,
                     workspace=0x20000, workspace_bytes=1 << 20)
    with pytest.raises(mira.MiraError) as e:
        mira.mira_moe_forward_noalloc(s, a, stream=1)
    assert e.value.code == -1 and "workspace" in mira.mira_last_error()
    a.workspace, a.workspace_bytes = None, 0
    big = next(T for T in range(16, 4096, 16)
               if mira.mira_workspace_bytes(s, T) > mira.MIRA_NOALLOC_SCRATCH_BYTES)
    a.n_tokens = big
    with pytest.raises(mira.MiraError) as e:
        mira.mira_moe_forward_noalloc(s, a, stream=1)
    assert e.value.code == -4 and "MIRA_NOALLOC_SCRATCH_BYTES" in mira.mira_last_error()
    assert mira.mira_workspace_bytes(s, 16) <= mira.MIRA_NOALLOC_SCRATCH_BYTES


def _stack_cfg(**kw):
    C, R = 256, 512
    base = dict(n_layers=4, n_hot=8, n_stage=4, max_tokens=8, slot_stride=mira.mira_packed_expert_bytes(C, R))
    base.update(kw)
    return mira.stack_config(**base), mira.MoEShape(C, R, 4, 2, 0, mira.MIRA_BF16)


@pytest.mark.parametrize("change,code", [
    (dict(n_layers=0), -2), (dict(n_hot=0, n_stage=0), -2), (dict(n_hot=-1), -2), (dict(max_tokens=0), -2),
    (dict(vram_mode=7), -1), (dict(lookahead=0), -1), (dict(stage_per_layer=0), -1),
    (dict(rb_interval=-1), -1), (dict(rb_interval=32, rb_probation=0), -1),
    (dict(slot_stride=1000), -2), (dict(slot_stride=256), -2),
])
def test_stack_create_rejects_bad_settings_before_the_gpu(change, code):
    """mira_stack_create checks its settings before any HIP call (these run
    without a GPU)."""
    cfg, shape = _stack_cfg(**change)
    with pytest.raises(mira.MiraError) as e:
        mira.mira_stack_create(cfg, shape, 0x100000, 0x2000, compute=1)
    assert e.value.code == code, mira.mira_last_error()


def test_stack_create_rejects_bad_shapes_and_pointers():
    cfg, shape = _stack_cfg()
    with pytest.raises(mira.MiraError) as e:
        mira.mira_stack_create(cfg, mira.MoEShape(256, 512, 255, 2, 2, mira.MIRA_BF16), 0x100000, 0x2000, compute=1)
    assert e.value.code == -2  # more than MIRA_MAX_EXPERTS experts per layer
    with pytest.raises(mira.MiraError) as e:
        mira.mira_stack_create(cfg, shape, None, 0x2000, compute=1)
    assert e.value.code == -1
    with pytest.raises(mira.MiraError) as e:
        mira.mira_stack_create(cfg, shape, 0x100080, 0x2000, compute=1)
    assert e.value.code == -3  # the slot pool must be 256-byte aligned
