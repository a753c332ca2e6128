"""GPU parity of the MoE expert step against the CPU oracle (small and
ragged shapes; full-size workloads are in test_gpu_fullsize.py).

Bars: packing, routing indices and the permutation bit-exact; the layer
output within rel-Frobenius 5e-3 and max-abs 2e-2 * rms(out)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_layer import EPS, Layer, act_dtype, assert_ffn_close, decode_rel_floor, run_and_check
from mira_inputs import CONFIGS, MoEConfig, predictor_weights, activations

pytestmark = pytest.mark.gpu


def _cfg(name, cid, **kw):
    return MoEConfig(name, cid, **kw)


SMALL_BF16 = _cfg("small_bf16", 101, T=16, C=128, E=8, k=2, R=192, zipf_s=1.2)
SMALL_FG = _cfg("small_fg", 102, T=16, C=128, E=64, k=6, R=128, S=2, zipf_s=1.0)
SMALL_F32 = _cfg("small_f32", 103, T=16, C=64, E=3, k=3, R=64, act="f32")


def test_pack_bit_exact_tiny(mira):
    lay = Layer(CONFIGS["tiny"])
    for e in range(4):
        ref = oracle.pack_expert(*lay.master(e), eps=EPS)
        assert np.array_equal(lay.slot_bytes(int(lay.table[e])), ref), e


def test_pack_bit_exact_bf16_input_and_padding(mira):
    C, R, n = 128, 256, 3
    g = torch.Generator().manual_seed(5)
    w = [torch.randn((n, *s), generator=g).mul_(0.03).to(torch.bfloat16) for s in ((R, C), (R, C), (C, R))]
    stride = mira.mira_packed_expert_bytes(C, R) + 1024
    out = torch.full((n * stride,), 0x5A, dtype=torch.uint8, device="cuda")
    mira.mira_pack_experts(mira.MoEShape(C, R, 1, 1), n, mira.MIRA_BF16, *(t.cuda() for t in w), EPS,
                           out, stride, 1)
    got = out.cpu().numpy().reshape(n, stride)
    for e in range(n):
        ref = oracle.pack_expert(*(t[e].float().numpy() for t in w), eps=EPS)
        assert np.array_equal(got[e, :ref.size], ref)
        assert not got[e, ref.size:].any()


@pytest.mark.parametrize("T", [16, 5])
def test_tiny_decode_path(mira, T):
    res, errs, _, _ = run_and_check(Layer(CONFIGS["tiny"], T=T))
    assert errs[0] < decode_rel_floor(T), errs  # the integer decode path keeps well inside the bar


# fp32 activations on the prefill path: x and H' travel as high and low bf16
# parts and both GEMMs run their k range over each, so the output is within a
# few 2^-16 of the oracle's instead of the 2^-9 of one bf16 rounding.
F32_PREFILL_REL = 1e-4


def test_tiny_prefill_path(mira):
    res, errs, _, _ = run_and_check(Layer(CONFIGS["tiny"]), flags=mira.MIRA_FLAG_FORCE_PREFILL)
    assert errs[0] < F32_PREFILL_REL, errs


@pytest.mark.parametrize("T", [40, 300])
def test_f32_prefill_two_passes_are_near_fp32(mira, T):
    # 300 tokens: several m-tiles per expert; C 128 / R 192: ragged n-tiles
    cfg = _cfg("f32_prefill", 107, T=T, C=128, E=8, k=2, R=192, zipf_s=1.2, act="f32")
    res, errs, _, _ = run_and_check(Layer(cfg))
    assert errs[0] < F32_PREFILL_REL, errs


def test_decode_and_prefill_paths_agree(mira):
    lay = Layer(SMALL_BF16)
    a = lay.run(mira.MIRA_FLAG_FORCE_DECODE)
    b = lay.run(mira.MIRA_FLAG_FORCE_PREFILL)
    assert np.array_equal(a["idx"], b["idx"]) and np.array_equal(a["order"], b["order"])
    assert_ffn_close(b["out"], a["out"], "prefill vs decode")


@pytest.mark.parametrize("T", [1, 2, 5, 6, 11, 15, 16, 17, 33, 64, 129])
def test_ragged_token_counts(mira, T):
    run_and_check(Layer(SMALL_BF16, T=T))


@pytest.mark.parametrize("T", [1, 7, 16, 40, 300])
def test_fine_grained_shape_small(mira, T):
    run_and_check(Layer(SMALL_FG, T=T))


# The largest expert count the interface takes (E + S = MIRA_MAX_EXPERTS):
# top-k over four 64-expert blocks per lane, 256 groups in the permutation
# and the decode descriptors (one-wave path beyond 64 pairs), and 16 expert
# tiles in the prefill router.  Decode routing equals prefill routing here too.
LARGE_E = _cfg("large_e", 106, T=16, C=128, E=255, k=8, R=64, S=1, zipf_s=1.0)


@pytest.mark.parametrize("T", [1, 9, 16, 40])
def test_largest_expert_count(mira, T):
    lay = Layer(LARGE_E, T=T)
    res, _, _, _ = run_and_check(lay)
    if T <= mira.MIRA_DECODE_MAX_TOKENS:
        pre = lay.run(mira.MIRA_FLAG_FORCE_PREFILL)
        for key in ("idx", "w", "logits", "counts", "offsets", "order"):
            assert np.array_equal(res[key], pre[key]), key


@pytest.mark.parametrize("T", [3, 24])
def test_softmax_over_all_experts_large_e(mira, T):
    # the selection over four 64-expert blocks per lane with the weights of a
    # softmax over all 255 experts: against the GPU's own exported logits
    # (exhaustive sort, fp64 softmax), so near ties cannot matter
    c = LARGE_E
    lay = Layer(c, T=T)
    res = lay.run(mira.MIRA_FLAG_SOFTMAX_ALL)
    assert res["status"][0] == 0
    for t in range(T):
        row = res["logits"][t].astype(np.float64)
        brute = sorted(range(c.E), key=lambda e: (-float(res["logits"][t, e]), e))[:c.k]
        assert res["idx"][t].tolist() == brute, t
        p = np.exp(row - row.max())
        p /= p.sum()
        assert np.max(np.abs(res["w"][t] - p[brute])) < 2e-6, t
    if T <= mira.MIRA_DECODE_MAX_TOKENS:
        pre = lay.run(mira.MIRA_FLAG_SOFTMAX_ALL | mira.MIRA_FLAG_FORCE_PREFILL)
        for key in ("idx", "w", "logits", "counts", "offsets", "order"):
            assert np.array_equal(res[key], pre[key]), key


@pytest.mark.parametrize("flags", [0, "decode", "prefill"])
def test_f32_activations_k_equals_E(mira, flags):
    f = {0: 0, "decode": mira.MIRA_FLAG_FORCE_DECODE, "prefill": mira.MIRA_FLAG_FORCE_PREFILL}[flags]
    res, errs, _, _ = run_and_check(Layer(SMALL_F32, T=13), flags=f)
    assert errs[0] < (F32_PREFILL_REL if flags == "prefill" else decode_rel_floor(13)), errs


def test_softmax_over_all_experts_flag(mira):
    lay = Layer(SMALL_BF16, T=9)
    res = lay.run(mira.MIRA_FLAG_SOFTMAX_ALL)
    o_x, o_wr, o_b = lay.oracle_inputs()
    lg = oracle.router_logits(o_x, o_wr, o_b)
    idx = oracle.topk_select(lg, SMALL_BF16.k)
    assert np.array_equal(res["idx"], idx)
    assert np.max(np.abs(res["w"] - oracle.combine_weights(lg, idx, norm_topk=False))) < 2e-5
    from gpu_layer import LazyBlobs
    ref = oracle.moe_forward(o_x, o_wr, o_b, LazyBlobs(lay), SMALL_BF16.k, SMALL_BF16.C, SMALL_BF16.R,
                             norm_topk=False)["out"]
    assert_ffn_close(res["out"], ref, "softmax-all")


def test_repeated_calls_bit_identical(mira):
    for flags in (0, mira.MIRA_FLAG_FORCE_PREFILL):
        lay = Layer(SMALL_FG, T=40)
        a, b = lay.run(flags), lay.run(flags)
        for k in a:
            assert np.array_equal(a[k], b[k]), k


def test_output_independent_of_slot_placement(mira):
    base = Layer(SMALL_BF16, T=24).run()
    perm = list(np.random.default_rng(0).permutation(SMALL_BF16.G))
    moved = Layer(SMALL_BF16, T=24, slot_order=perm, spare_slots=3).run()
    assert np.array_equal(base["out"], moved["out"])
    assert np.array_equal(base["order"], moved["order"])


def test_non_resident_selected_expert_sets_status(mira):
    lay = Layer(SMALL_BF16, T=16, resident=[1, 2, 3, 4, 5, 6, 7])  # expert 0 (most popular) absent
    res = lay.run()
    assert res["counts"][0] > 0
    assert res["status"][0] & 1
    lay2 = Layer(SMALL_BF16, T=16)
    lay2.table[0] = 99  # beyond n_slots: ignored, flagged
    res2 = lay2.run()
    assert res2["status"][0] & 2


class _ZeroExpert:
    """Oracle blobs with one expert replaced by an all-zero blob (sigma = 0,
    q = 0), whose FFN output is exactly zero: the oracle's layer output with
    that expert's term left out and every other term and weight unchanged."""

    def __init__(self, blobs, missing, nbytes):
        self.blobs, self.missing, self.nbytes = blobs, missing, nbytes

    def __len__(self):
        return len(self.blobs)

    def __getitem__(self, e):
        return np.zeros(self.nbytes, dtype=np.uint8) if e == self.missing else self.blobs[e]


@pytest.mark.parametrize("T,path", [(16, "decode"), (16, "prefill"), (150, "prefill"), (150, "auto")])
def test_missing_selected_expert_contributes_nothing(mira, T, path):
    """A selected expert whose slot is -1 sets status bit 0 and its term is
    missing from out (every other term present), on both expert paths.  The
    workspace starts as NaN bytes, so a combine that read the missing
    expert's never-written rows would show."""
    from gpu_layer import LazyBlobs, check_routing
    flags = {"decode": mira.MIRA_FLAG_FORCE_DECODE, "prefill": mira.MIRA_FLAG_FORCE_PREFILL,
             "auto": 0}[path]
    cfg = SMALL_BF16
    lay = Layer(cfg, T=T, resident=[1, 2, 3, 4, 5, 6, 7])
    res = lay.run(flags, ws_fill=0xFF)
    assert res["counts"][0] > 0
    assert res["status"][0] == 1
    o_x, o_wr, o_b = lay.oracle_inputs()
    o_logits = oracle.router_logits(o_x, o_wr, o_b)
    assert not check_routing(res, lay, o_logits)  # no near ties at this seed
    blobs = _ZeroExpert(LazyBlobs(lay), 0, lay.stride)
    ref = oracle.moe_forward(o_x, o_wr, o_b, blobs, cfg.k, cfg.C, cfg.R)["out"]
    assert_ffn_close(res["out"], ref, f"missing expert 0, {path}")


# The down GEMM of the prefill path splits its contraction R into KS chunks
# (KS <= R/4096, at most 4) and the combine sums the chunk partials in order.
# With C = 256 the layer has one 512-row output tile, so at 300 tokens over
# 4 experts (at most 8 m-tiles of 128) the grid's cost rule picks the largest
# split: KS = 2 at R = 8192 and KS = 4 at R = 16384.  Every row is checked.
KSPLIT_R8K = _cfg("ksplit_r8k", 107, T=300, C=256, E=4, k=2, R=8192, zipf_s=1.2)
KSPLIT_R16K = _cfg("ksplit_r16k", 108, T=300, C=256, E=4, k=2, R=16384, zipf_s=1.2)


@pytest.mark.parametrize("cfg", [KSPLIT_R8K, KSPLIT_R16K], ids=lambda c: c.name)
def test_prefill_down_k_split_all_rows(mira, cfg):
    lay = Layer(cfg)
    res, errs, _, _ = run_and_check(lay, flags=mira.MIRA_FLAG_FORCE_PREFILL)
    print(f"{cfg.name}: rel_fro={errs[0]:.2e} max_abs/rms={errs[1]:.2e}")


def test_two_phase_demand_fetch_through_pinned_store(mira):
    """Route, read the counts, stage the missing experts from pinned host
    memory into spare slots, then run the experts: bit-identical to the
    all-resident call."""
    cfg = SMALL_BF16
    full = Layer(cfg, T=16).run()
    lay = Layer(cfg, T=16, resident=[4, 5, 6, 7], spare_slots=4)
    stride = lay.stride
    host = torch.empty((cfg.E, stride), dtype=torch.uint8, pin_memory=True)
    sh = mira.MoEShape(cfg.C, cfg.R, 1, 1)
    for e in range(cfg.E):
        wg, wu, wd = (np.ascontiguousarray(t) for t in lay.master(e))
        mira.mira_pack_experts(sh, 1, mira.MIRA_F32, wg.ctypes.data, wu.ctypes.data, wd.ctypes.data, EPS,
                               host[e], stride, 0)
    copy = torch.cuda.Stream()
    compute = torch.cuda.current_stream()

    def fetch(r):
        counts = r["counts"].cpu().numpy()
        table = lay.table.cpu().numpy()
        free = [s for s in range(lay.n_slots) if s not in set(table.tolist())]
        ev = torch.cuda.Event()
        for e in range(cfg.E):
            if counts[e] > 0 and table[e] < 0:
                slot = free.pop(0)
                mira.mira_stage_expert(lay.pool, stride, slot, host[e], stride, copy, None)
                mira.mira_set_slot(lay.table, e, slot, copy)
        ev.record(copy)
        compute.wait_event(ev)

    res = lay.run(two_phase=True, between=fetch)
    assert res["status"][0] == 1  # the route phase saw the misses
    assert np.array_equal(res["out"], full["out"])
    assert np.array_equal(res["idx"], full["idx"])


def test_stage_copy_is_byte_exact(mira):
    n = 3 * 1024 * 1024 + 512
    src = torch.randint(0, 256, (n,), dtype=torch.uint8).pin_memory()
    pool = torch.zeros(2 * n + 256, dtype=torch.uint8, device="cuda")
    ev = torch.cuda.Event()
    s = torch.cuda.Stream()
    mira.mira_stage_expert(pool, n + 256, 1, src, n, s, ev)
    ev.synchronize()
    assert torch.equal(pool[n + 256:2 * n + 256].cpu(), src)
    assert not pool[:n + 256].any()


def test_predictor_matches_oracle(mira):
    cfg = CONFIGS["beam_stack"]
    x = activations(cfg, 3, "cpu", T=16)
    w1, b1, w2, b2 = predictor_weights(cfg, 3, "cpu")
    b1 = torch.randn(b1.shape, generator=torch.Generator().manual_seed(1)) * 0.1
    p = mira.PredShape(cfg.C, cfg.pred_hidden, cfg.E, cfg.pred_group, mira.MIRA_BF16)
    ws = torch.empty(mira.mira_predict_workspace_bytes(p, 16), dtype=torch.uint8, device="cuda")
    scores = torch.zeros((2, cfg.E), dtype=torch.float32, device="cuda")
    mira.mira_predict(p, x.cuda(), 16, w1.cuda(), b1.cuda(), w2.cuda(), b2.cuda(), scores, ws, ws.numel())
    torch.cuda.synchronize()
    ref = oracle.predictor_scores(x.float().numpy(), cfg.pred_group, w1.float().numpy(), b1.numpy(),
                                  w2.float().numpy(), b2.numpy())
    assert np.max(np.abs(scores.cpu().numpy() - ref)) < 1e-4


def test_zero_tokens_is_a_noop(mira):
    lay = Layer(SMALL_BF16, T=4)
    s = lay.shape()
    a = mira.MoEArgs(n_tokens=0)
    mira.mira_moe_forward(s, a)
    torch.cuda.synchronize()


# Small decode calls: the one-shot call and the two-phase API (route, then
# experts) give bit-identical results, and the decode routing equals the
# prefill path's (both reduce the same 16 k-range slices in the same order).
@pytest.mark.parametrize("cfg,T", [(SMALL_BF16, 1), (SMALL_BF16, 3), (SMALL_BF16, 5), (SMALL_FG, 1),
                                   (SMALL_FG, 4), (SMALL_F32, 2), (SMALL_F32, 5)])
def test_decode_one_shot_matches_two_phase_and_prefill_routing(mira, cfg, T):
    lay = Layer(cfg, T=T)
    one = lay.run()
    split = lay.run(two_phase=True)
    for key in one:
        assert np.array_equal(one[key], split[key]), key
    pre = lay.run(mira.MIRA_FLAG_FORCE_PREFILL)
    for key in ("idx", "w", "logits", "counts", "offsets", "order"):
        assert np.array_equal(one[key], pre[key]), key
    run_and_check(lay, res=one)


@pytest.mark.parametrize("cfg,T", [(SMALL_BF16, 1), (SMALL_BF16, 3), (SMALL_BF16, 5), (SMALL_FG, 1),
                                   (SMALL_F32, 2)])
def test_decode_results_independent_of_workspace_contents(mira, cfg, T):
    """Nothing in the workspace needs to start in a given state: a workspace
    of 0xFF bytes, one of 0xA5, one of zeros and the same workspace reused
    give bit-identical results that match the oracle."""
    lay = Layer(cfg, T=T)
    ref = lay.run(ws_fill=0x00)
    for fill in (0xFF, 0xA5, None):
        got = lay.run(ws_fill=fill)
        for key in ref:
            assert np.array_equal(got[key], ref[key]), (fill, key)
    run_and_check(lay, res=ref)


def test_predictor_groups_are_independent(mira):
    """A group's scores do not depend on the other groups of the call (1, 4
    or 5 groups give bit-identical scores for the groups they share), from a
    workspace of 0xFF bytes and when the workspace is reused; all match the
    oracle.  Calls of up to 4 groups pool inside the first layer's kernel and
    5 groups take the separate pooling kernel, so this also checks that both
    give the same bits."""
    cfg = CONFIGS["beam_stack"]
    x = activations(cfg, 4, "cpu", T=40)
    w1, b1, w2, b2 = predictor_weights(cfg, 4, "cpu")
    b1 = torch.randn(b1.shape, generator=torch.Generator().manual_seed(2)) * 0.1
    b2 = torch.randn(b2.shape, generator=torch.Generator().manual_seed(3)) * 0.1
    dev = [t.cuda() for t in (w1, b1, w2, b2)]
    p = mira.PredShape(cfg.C, cfg.pred_hidden, cfg.E, cfg.pred_group, mira.MIRA_BF16)
    out = {}
    for T in (32, 40, 8):
        ws = torch.full((mira.mira_predict_workspace_bytes(p, T),), 0xFF, dtype=torch.uint8, device="cuda")
        sc = torch.zeros((T // cfg.pred_group, cfg.E), dtype=torch.float32, device="cuda")
        for _ in range(2):  # the second call reuses the workspace
            mira.mira_predict(p, x[:T].cuda(), T, *dev[:2], *dev[2:], sc, ws, ws.numel())
        torch.cuda.synchronize()
        out[T] = sc.cpu().numpy()
        ref = oracle.predictor_scores(x[:T].float().numpy(), cfg.pred_group, w1.float().numpy(), b1.numpy(),
                                      w2.float().numpy(), b2.numpy())
        assert np.max(np.abs(out[T] - ref)) < 1e-4, T
    assert np.array_equal(out[32], out[40][:4])
    assert np.array_equal(out[8], out[40][:1])
