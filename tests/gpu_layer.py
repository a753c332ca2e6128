"""Build one synthetic MoE layer on the GPU (experts packed into a slot pool
by the library) and the oracle's view of the same seeded inputs.

The oracle always packs from the fp32 master weights itself; nothing it uses
comes from the library."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2609_38090_amd as mira
from mira_inputs import activations, expert_weights, router_bias, router_weights

EPS = 1e-8
FFN_REL_FRO = 5e-3       # relative Frobenius error bar of the layer output
FFN_MAX_ABS_RMS = 2e-2   # max-abs error bar, in units of rms(out)
NEAR_TIE = 1e-4          # logit gap below which a top-k decision is ambiguous


def decode_rel_floor(T):
    """Relative Frobenius error the integer decode path keeps to, well inside
    FFN_REL_FRO: the int8 matrix-core sums are exact and the rounding is the
    fixed point of x (22 bits of the token's maximum) and of H' (22 bits of its
    64-row block maximum up to 5 tokens; 14 bits above, where H' is carried as
    two digits so an operand holds 8 tokens).  At 14 bits one H' entry is off
    by at most 2^-14 of its block maximum; the outputs of these inputs then
    differ by about 1e-4 of their norm."""
    return 1e-4 if T <= 5 else 1e-3


def act_dtype(cfg):
    return mira.MIRA_F32 if cfg.act == "f32" else mira.MIRA_BF16


def gen_device(cfg):
    return "cpu" if cfg.C * cfg.R <= (1 << 22) else "cuda"


def to_np(t):
    return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.detach().cpu().numpy()


class LazyBlobs:
    """blobs[e] = oracle.pack_expert of expert e's master weights, computed on demand."""

    def __init__(self, layer):
        self.layer = layer
        self.cache = {}

    def __len__(self):
        return self.layer.cfg.E

    def __getitem__(self, e):
        if e not in self.cache:
            self.cache[e] = self.layer.oracle_pack(*self.layer.master(e))
        return self.cache[e]


class Layer:
    def __init__(self, cfg, layer=0, resident=None, spare_slots=0, T=None, slot_order=None,
                 device="cuda", fmt="int8"):
        self.cfg, self.layer, self.device, self.fmt = cfg, layer, device, fmt
        self.fflag = mira.MIRA_FLAG_INT4 if fmt == "int4" else 0
        self.T = cfg.T if T is None else T
        self.stride = (mira.mira_packed_expert_bytes_int4(cfg.C, cfg.R) if fmt == "int4"
                       else mira.mira_packed_expert_bytes(cfg.C, cfg.R))
        gd = gen_device(cfg)
        self.x = activations(cfg, layer, gd, T=self.T).to(device)
        self.wr = router_weights(cfg, layer, gd).to(device)
        b = router_bias(cfg, layer)
        self.bias = b.to(device) if b is not None else None
        resident = list(range(cfg.G)) if resident is None else list(resident)
        if slot_order is not None:
            resident = [resident[i] for i in slot_order]
        self.resident = resident
        self.n_slots = max(1, len(resident) + spare_slots)
        self.pool = torch.zeros(self.n_slots * self.stride, dtype=torch.uint8, device=device)
        table = [-1] * cfg.G
        self.shape_pack = mira.MoEShape(cfg.C, cfg.R, 1, 1, flags=self.fflag)
        for slot, e in enumerate(resident):
            self.pack_into(e, slot)
            table[e] = slot
        self.table = torch.tensor(table, dtype=torch.int32, device=device)
        torch.cuda.synchronize()

    def master_dev(self, e):
        return expert_weights(self.cfg, self.layer, e, gen_device(self.cfg))

    def master(self, e):
        return tuple(t.cpu().numpy() for t in self.master_dev(e))

    def pack_into(self, e, slot):
        wg, wu, wd = (t.to(self.device) for t in self.master_dev(e))
        mira.mira_pack_experts(self.shape_pack, 1, mira.MIRA_F32, wg, wu, wd, EPS,
                               self.pool[slot * self.stride:], self.stride, 1)

    def slot_bytes(self, slot):
        return self.pool[slot * self.stride:(slot + 1) * self.stride].cpu().numpy()

    def shape(self, flags=0):
        c = self.cfg
        return mira.MoEShape(c.C, c.R, c.E, c.k, c.S, act_dtype(c), flags | self.fflag)

    def run(self, flags=0, two_phase=False, between=None, stream=None, sync=True, ws_fill=None):
        """One layer call; returns the outputs as numpy arrays, or with
        sync=False the device tensors (the call only queued on stream).
        ws_fill: a byte value the workspace is filled with first (0xFF makes
        every fp32 word of it a NaN, so a read of an unwritten region shows)."""
        c, T, dev = self.cfg, self.T, self.device
        s = self.shape(flags)
        P = T * c.k + c.S * T
        ws = torch.empty(mira.mira_workspace_bytes(s, T), dtype=torch.uint8, device=dev)
        if ws_fill is not None:
            ws.fill_(ws_fill)
        r = dict(
            out=torch.full((T, c.C), float("nan"), dtype=torch.float32, device=dev),
            idx=torch.full((T, c.k), -7, dtype=torch.int32, device=dev),
            w=torch.zeros((T, c.k), dtype=torch.float32, device=dev),
            logits=torch.zeros((T, c.E), dtype=torch.float32, device=dev),
            counts=torch.zeros((c.G,), dtype=torch.int32, device=dev),
            status=torch.full((1,), -1, dtype=torch.int32, device=dev),
            offsets=torch.zeros((c.G + 1,), dtype=torch.int32, device=dev),
            order=torch.full((max(P, 1),), -1, dtype=torch.int32, device=dev),
        )
        a = mira.MoEArgs(x=self.x, n_tokens=T, n_slots=self.n_slots, w_router=self.wr,
                         router_bias=self.bias, slot_table=self.table, slot_pool=self.pool,
                         slot_stride=self.stride, out=r["out"], topk_idx=r["idx"], topk_weight=r["w"],
                         logits=r["logits"], expert_counts=r["counts"], status=r["status"],
                         expert_offsets=r["offsets"], pair_order=r["order"], workspace=ws,
                         workspace_bytes=ws.numel())
        if two_phase:
            mira.mira_moe_route(s, a, stream)
            if between is not None:
                between(r)
            mira.mira_moe_experts(s, a, stream)
        else:
            mira.mira_moe_forward(s, a, stream)
        if not sync:
            r["_ws"] = ws  # keep the workspace alive until the caller synchronizes
            return r
        torch.cuda.synchronize()
        return {k: v.cpu().numpy() for k, v in r.items()}

    # ---- oracle side ------------------------------------------------------
    def oracle_inputs(self):
        x = to_np(self.x).astype(np.float64)
        wr = to_np(self.wr).astype(np.float64)
        b = None if self.bias is None else self.bias.cpu().numpy().astype(np.float64)
        return x, wr, b

    def oracle_pack(self, wg, wu, wd):
        """The oracle's own packing of master weights, in this layer's format."""
        if self.fmt == "int4":
            return oracle.pack_expert_int4(wg, wu, wd, eps=EPS)
        return oracle.pack_expert(wg, wu, wd, eps=EPS)

    def shared_blobs(self):
        c = self.cfg
        return [self.oracle_pack(*self.master(c.E + s)) for s in range(c.S)]


def ffn_error(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = got - ref
    rms = np.sqrt(np.mean(ref ** 2))
    rel_fro = np.linalg.norm(d) / max(np.linalg.norm(ref), 1e-300)
    max_abs = np.max(np.abs(d)) / max(rms, 1e-300) if d.size else 0.0
    return rel_fro, max_abs


def assert_ffn_close(got, ref, what=""):
    rel_fro, max_abs = ffn_error(got, ref)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    assert rel_fro <= FFN_REL_FRO and max_abs <= FFN_MAX_ABS_RMS, \
        f"{what}: rel_fro={rel_fro:.3e} max_abs/rms={max_abs:.3e}"
    return rel_fro, max_abs


def topk_candidates(logits_row, k, delta=NEAR_TIE):
    """Every expert set an equally valid rounding could select: experts clearly
    above the k-th logit (by more than delta) are required, experts within
    delta of it fill the remaining places in every combination."""
    import itertools
    v = np.sort(logits_row)[::-1]
    vk = v[k - 1]
    must = [e for e in range(len(logits_row)) if logits_row[e] > vk + delta]
    may = [e for e in range(len(logits_row)) if abs(logits_row[e] - vk) <= delta and e not in must]
    return [tuple(sorted(must + list(c))) for c in itertools.combinations(may, k - len(must))]


def check_routing(res, lay, o_logits):
    """Routing outputs against the oracle; returns the near-tie tokens.

    Outside the near-tie set the GPU must reproduce the oracle's selection,
    weights, counts and permutation exactly (weights to fp32 rounding).  On
    near-tie tokens the selection must be one of the oracle's candidates and
    the rest must be consistent with it."""
    c, T = lay.cfg, lay.T
    g_logits = res["logits"].astype(np.float64)
    scale = np.maximum(1.0, np.abs(o_logits))
    assert np.max(np.abs(g_logits - o_logits) / scale) < 2e-5
    # top-k is exactly the exhaustive sort of the GPU's own logits
    for t in range(T):
        brute = sorted(range(c.E), key=lambda e: (-float(res["logits"][t, e]), e))[:c.k]
        assert res["idx"][t].tolist() == brute, t
    o_idx = oracle.topk_select(o_logits, c.k)
    o_w = oracle.combine_weights(o_logits, o_idx)
    ties = set(oracle.near_tie_tokens(o_logits, c.k, NEAR_TIE).tolist())
    for t in range(T):
        if t in ties:
            assert tuple(sorted(res["idx"][t].tolist())) in topk_candidates(o_logits[t], c.k), t
            sel = res["logits"][t, res["idx"][t]].astype(np.float64)
            e = np.exp(sel - sel.max())
            assert np.max(np.abs(res["w"][t] - e / e.sum())) < 2e-6, t
        else:
            assert res["idx"][t].tolist() == o_idx[t].tolist(), t
            assert np.max(np.abs(res["w"][t] - o_w[t])) < 2e-5, t
    # counts, offsets and the permutation: the stable grouping of the GPU's
    # selection (brute force), and the oracle's own when no token is ambiguous
    P = T * c.k + c.S * T
    group = np.concatenate([res["idx"].reshape(-1), np.repeat(np.arange(c.E, c.G), T)]).astype(np.int64)
    counts = np.bincount(group, minlength=c.G)
    assert res["counts"].tolist() == counts.tolist()
    assert res["offsets"].tolist() == [0] + np.cumsum(counts).tolist()
    assert res["order"][:P].tolist() == sorted(range(P), key=lambda p: (group[p], p))
    if not ties:
        oc, oo, op, _ = oracle.permute_pairs(o_idx, c.E, c.S)
        assert res["counts"].tolist() == oc.tolist()
        assert res["order"][:P].tolist() == op.tolist()
    return ties


def run_and_check(lay, flags=0, tokens=None, res=None, blobs=None):
    """Run (or take) one layer call and check it against the oracle.

    Routing is checked by check_routing.  The output rows of `tokens` (all by
    default) are compared with the oracle's: outside the near-tie set under
    the oracle's own selection; on a near-tie token (whose selection
    check_routing has found to be one of the oracle's candidates) under the
    selection the GPU exported for that token, so the output must be the one
    of exactly the experts reported in topk_idx."""
    c = lay.cfg
    if res is None:
        res = lay.run(flags)
    assert res["status"][0] == 0
    o_x, o_wr, o_b = lay.oracle_inputs()
    o_logits = oracle.router_logits(o_x, o_wr, o_b)
    ties = check_routing(res, lay, o_logits)
    tokens = list(range(lay.T)) if tokens is None else list(tokens)
    blobs = LazyBlobs(lay) if blobs is None else blobs
    shared = lay.shared_blobs()
    plain = [t for t in tokens if t not in ties]
    tied = [t for t in tokens if t in ties]
    ref = np.zeros((len(tokens), c.C))
    if plain:
        o = oracle.moe_forward(o_x, o_wr, o_b, blobs, c.k, c.C, c.R, shared_blobs=shared, tokens=plain,
                               fmt=lay.fmt)
        for i, t in enumerate(plain):
            ref[tokens.index(t)] = o["out"][i]
    if tied:
        gpu_idx = oracle.topk_select(o_logits, c.k)
        for t in tied:
            gpu_idx[t] = res["idx"][t]
        o = oracle.moe_forward(o_x, o_wr, o_b, blobs, c.k, c.C, c.R, shared_blobs=shared, idx=gpu_idx,
                               tokens=tied, fmt=lay.fmt)
        for i, t in enumerate(tied):
            ref[tokens.index(t)] = o["out"][i]
    got = res["out"][tokens]
    errs = assert_ffn_close(got, ref, f"{c.name} {lay.fmt} flags={flags}")
    return res, errs, blobs, ties
