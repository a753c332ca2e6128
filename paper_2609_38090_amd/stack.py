"""A stack of MoE layers over a device expert pool with HOT and STAGE slots.

Paper sections IV-C (HOT and STAGE regions of the expert cache), IV-D
(telemetry-driven rebalancing of the HOT set), IV-E (predictive staging of
layer l+2's experts on a copy stream) and IV-F (the staging copies overlap the
compute stream).  This module is the host-side bookkeeping of a decode step
through L layers; every byte still moves through the library:
mira_moe_route / mira_moe_experts run a layer, mira_predict (the MLP head) or
mira_predict_mixture (the MixtureHead, fed by the layer's router logits and
selections) scores layer l+2's experts, mira_stage_expert copies a packed expert from pinned host
memory into a slot on the copy stream, and mira_set_slot updates a layer's
slot table in stream order.

HOT and STAGE are labels on slots of one pool: each HOT slot holds one expert
of one layer until the rebalancer evicts it; STAGE slots are the prefetch
window.  Policy, per layer l of a step:
  1. route layer l; read which experts its tokens selected and how many tokens
     each received;
  2. every selected expert is served from its HOT slot, from a STAGE slot
     filled earlier (the compute stream waits for that copy), or by a demand
     copy into a free STAGE slot (a CPU-served miss); the tokens and the tier
     go to the layer's telemetry;
  3. run the experts of layer l;
  4. prefetch controller: choose experts of layer l+2 (mode "predict": the
     `stage_per_layer` best-scored experts of the predictor head; "oracle"
     (oracle prefetch, a perfect predictor): every expert layer l+2 will
     select, taken from that layer's routing as this library computed it on
     an earlier pass, an upper bound; "demand": none); an
     expert already in HOT or STAGE is a skipped prefetch, a repeated request
     for the same (expert, layer) issues no second copy, and when no STAGE slot
     is free the prefetch is declined;
  5. when the layer's telemetry window is full, the rebalancer swaps a bounded
     number of HOT experts for candidates; a candidate held in a STAGE slot is
     promoted by relabelling that slot, otherwise it is copied from the CPU
     store into the evicted expert's slot.
STAGE slots whose layer has passed are free again; in "small" VRAM mode they
are released right after their layer, in "large" mode they keep their expert
(a later step may hit it) until a copy needs the slot.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

from . import _binding as mira
from .policy import Rebalancer, Telemetry


@dataclass
class StepStats:
    hot_hits: int = 0
    stage_hits: int = 0
    misses: int = 0
    prefetches: int = 0
    prefetch_cached: int = 0     # predicted expert already in HOT or STAGE
    prefetch_declined: int = 0   # no STAGE slot free
    swaps: int = 0               # HOT rebalancing swaps
    promote_copies: int = 0      # swaps whose expert came from the CPU store
    h2d_bytes: int = 0
    copy_ms: float = 0.0         # summed durations of the copies (copy stream)
    stall_ms: float = 0.0        # time the compute stream waited for copies
    wall_ms: float = 0.0
    hot_tokens: int = 0          # tokens served by HOT / STAGE / CPU-copied experts
    stage_tokens: int = 0
    cpu_tokens: int = 0

    def add(self, o: "StepStats"):
        for k in self.__dataclass_fields__:
            setattr(self, k, getattr(self, k) + getattr(o, k))


@dataclass
class LayerData:
    x: torch.Tensor             # [T][C] activations of the layer (teacher forcing)
    w_router: torch.Tensor      # [E][C]
    bias: torch.Tensor | None   # [E] fp32
    hot: list                   # experts resident in HOT slots at the start
    host: dict = field(default_factory=dict)  # expert -> pinned packed blob (experts not HOT at the start)
    pred: object = None         # head scoring layer l+2: (w1, b1, w2, b2) of the MLP head,
                                # or mira.MixtureWeights of a MixtureHead


class ExpertStack:
    """L layers of one MoE shape sharing a slot pool: one HOT slot per resident
    expert of every layer, then n_stage STAGE slots."""

    def __init__(self, shape: mira.MoEShape, tokens: int, layers: list, stride: int,
                 n_stage: int, pred_shape=None, device="cuda",
                 vram_mode: str = "large", rebalancer: Rebalancer | None = None):
        if vram_mode not in ("small", "large"):
            raise ValueError("vram_mode must be 'small' or 'large'")
        self.shape, self.T, self.layers, self.stride = shape, tokens, layers, stride
        self.E = shape.n_experts
        self.device = device
        n_hot = sum(len(ld.hot) for ld in layers)
        need = max(self.E + shape.n_shared - len(ld.hot) for ld in layers)
        if n_stage < need:
            raise ValueError(f"{n_stage} STAGE slots cannot hold the {need} non-resident experts "
                             "one layer may select")
        self.n_hot, self.n_stage = n_hot, n_stage
        self.n_slots = n_hot + n_stage
        self.vram_mode, self.rebalancer = vram_mode, rebalancer
        self.pool = torch.zeros(self.n_slots * stride, dtype=torch.uint8, device=device)
        self.tables = torch.full((len(layers), self.E), -1, dtype=torch.int32, device=device)
        self.role = ["hot"] * n_hot + ["stage"] * n_stage
        self.held = [None] * self.n_slots     # (layer, expert) in the slot
        self.ready = [None] * self.n_slots    # event of the copy that filled the slot
        self.age = [0] * self.n_slots
        self.clock = 0
        self.hot_slot = []                    # per layer: expert -> HOT slot
        self.table_set = []                   # per layer: experts whose table entry is valid
        s = 0
        for l, ld in enumerate(layers):
            m = {}
            for e in ld.hot:
                m[e] = s
                self.held[s] = (l, e)
                self.tables[l, e] = s
                s += 1
            self.hot_slot.append(m)
            self.table_set.append(set(m))
        self.telemetry = [Telemetry(self.E) for _ in layers]
        self.ws = torch.empty(mira.mira_workspace_bytes(shape, tokens), dtype=torch.uint8, device=device)
        self.out = torch.empty((tokens, shape.hidden), dtype=torch.float32, device=device)
        self.idx = torch.empty((tokens, shape.top_k), dtype=torch.int32, device=device)
        self.counts = torch.zeros((self.E + shape.n_shared,), dtype=torch.int32, device=device)
        self.counts_h = torch.zeros_like(self.counts, device="cpu").pin_memory()
        self.status = torch.zeros((1,), dtype=torch.int32, device=device)
        self.pred_shape, self.mixture, self.logits = None, False, None
        self.set_predictor(pred_shape)
        self.compute = torch.cuda.current_stream(device)
        self.copy = torch.cuda.Stream(device)  # default priority
        self.side = torch.cuda.Stream(device)  # predictor heads, beside the experts (default priority)

    def set_predictor(self, pred_shape, heads=None):
        """Select the predictor head: a mira.PredShape (MLP heads) or a
        mira.MixtureShape (MixtureHeads, which also read the router logits).
        heads, if given, replaces LayerData.pred of every layer."""
        if heads is not None:
            for ld, h in zip(self.layers, heads):
                ld.pred = h
        self.pred_shape = pred_shape
        self.mixture = isinstance(pred_shape, mira.MixtureShape)
        self.logits = (torch.empty((self.T, self.E), dtype=torch.float32, device=self.device)
                       if self.mixture else None)
        if pred_shape is not None:
            ws = (mira.mira_mixture_workspace_bytes(pred_shape, self.T) if self.mixture
                  else mira.mira_predict_workspace_bytes(pred_shape, self.T))
            self.pws = torch.empty(max(ws, 256), dtype=torch.uint8, device=self.device)
            self.scores = torch.empty((self.T // pred_shape.group, pred_shape.n_out), dtype=torch.float32,
                                      device=self.device)
            self.scores_h = torch.zeros(self.scores.shape, dtype=torch.float32).pin_memory()

    def _predict(self, l: int):
        """Queue layer l's predictor head and the copy of its scores to the
        host on the side stream."""
        ld = self.layers[l]
        if self.mixture:
            mira.mira_predict_mixture(self.pred_shape, ld.pred, ld.x, self.logits, self.idx, self.T,
                                      self.scores, None, self.pws, self.pws.numel(), self.side)
        else:
            w1p, b1p, w2p, b2p = ld.pred
            mira.mira_predict(self.pred_shape, ld.x, self.T, w1p, b1p, w2p, b2p, self.scores, self.pws,
                              self.pws.numel(), self.side)
        with torch.cuda.stream(self.side):
            self.scores_h.copy_(self.scores, non_blocking=True)

    def args(self, l: int) -> mira.MoEArgs:
        ld = self.layers[l]
        return mira.MoEArgs(x=ld.x, n_tokens=self.T, n_slots=self.n_slots, w_router=ld.w_router,
                            router_bias=ld.bias, slot_table=self.tables[l], slot_pool=self.pool,
                            slot_stride=self.stride, out=self.out, topk_idx=self.idx,
                            logits=self.logits, expert_counts=self.counts, status=self.status, workspace=self.ws,
                            workspace_bytes=self.ws.numel())

    def hot_set(self, l: int) -> set:
        return set(self.hot_slot[l])

    # ---- slots -------------------------------------------------------------
    def _staged(self, l, e):
        for i in range(self.n_slots):
            if self.role[i] == "stage" and self.held[i] == (l, e):
                return i
        return -1

    def _free_stage(self, cur_layer, for_demand):
        """A STAGE slot for a copy made while layer cur_layer is current: a free
        slot, else the oldest slot of a passed layer; a demand copy may also
        take the oldest prefetch for a later layer (that prefetch is lost).
        Slots holding the current layer's experts are never taken."""
        stage = [i for i in range(self.n_slots) if self.role[i] == "stage"]
        cands = [i for i in stage if self.held[i] is None or self.held[i][0] < cur_layer]
        if not cands and for_demand:
            cands = [i for i in stage if self.held[i][0] > cur_layer]
        if not cands:
            return -1
        free = [i for i in cands if self.held[i] is None]
        return free[0] if free else min(cands, key=lambda i: self.age[i])

    def _copy_in(self, slot, l, e, st: StepStats, copy_events):
        """Copy expert e of layer l from the CPU store into `slot` (copy stream)."""
        # the slot's previous expert may still be read by kernels queued on
        # the compute stream: the copy waits for them
        done_before = torch.cuda.Event()
        done_before.record(self.compute)
        self.copy.wait_event(done_before)
        t0, t1, done = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
                        torch.cuda.Event())
        t0.record(self.copy)
        blob = self.layers[l].host[e]
        mira.mira_stage_expert(self.pool, self.stride, slot, blob, blob.numel(), self.copy, None)
        t1.record(self.copy)
        done.record(self.copy)
        copy_events.append((t0, t1))
        st.h2d_bytes += blob.numel()
        self.held[slot] = (l, e)
        self.ready[slot] = done
        self.clock += 1
        self.age[slot] = self.clock

    def _stage(self, l, e, cur_layer, for_demand, st, copy_events):
        i = self._free_stage(cur_layer, for_demand)
        if i < 0:
            if for_demand:  # cannot happen with n_stage >= experts per layer outside HOT
                raise RuntimeError("no STAGE slot free for a demand copy")
            st.prefetch_declined += 1
            return -1
        self._copy_in(i, l, e, st, copy_events)
        return i

    def _use(self, l, e, slot, stall_events):
        """Make layer l's table point expert e at `slot` before its experts run."""
        if self.ready[slot] is not None:
            b, c = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            b.record(self.compute)
            self.compute.wait_event(self.ready[slot])
            c.record(self.compute)
            stall_events.append((b, c))
            if self.role[slot] == "hot":
                self.ready[slot] = None  # a HOT copy is waited for once
        if e not in self.table_set[l]:
            mira.mira_set_slot(self.tables[l], e, slot, self.compute)
            self.table_set[l].add(e)

    def _unset(self, l, e):
        if e in self.table_set[l]:
            mira.mira_set_slot(self.tables[l], e, -1, self.compute)
            self.table_set[l].discard(e)

    def _rebalance(self, l, st, copy_events):
        tel = self.telemetry[l]
        for sw in self.rebalancer.plan(tel, self.hot_set(l)):
            sv = self.hot_slot[l].pop(sw.evict)
            self._unset(l, sw.evict)
            sc = self._staged(l, sw.promote)
            if sc >= 0:
                # the staged copy becomes the HOT copy; the evicted slot joins STAGE
                self._unset(l, sw.promote)
                self.role[sc], self.role[sv] = "hot", "stage"
                self.held[sv], self.ready[sv] = None, None
                self.hot_slot[l][sw.promote] = sc
            else:
                self._copy_in(sv, l, sw.promote, st, copy_events)
                self.hot_slot[l][sw.promote] = sv
                st.promote_copies += 1
            st.swaps += 1
        tel.close_window()

    # ---- one decode step through every layer ------------------------------
    def step(self, mode: str = "predict", stage_per_layer: int = 2, true_idx=None,
             on_layer=None) -> StepStats:
        """One decode step through every layer.  true_idx[l] (the routing of
        layer l, from an earlier pass of this stack) is needed by mode
        "oracle"; on_layer(l, out), if given, is
        called after layer l's experts are queued (out is reused by the next
        layer, so copy it on the compute stream)."""
        st = StepStats()
        L = len(self.layers)
        copy_events, stall_events = [], []
        w0, w1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        w0.record(self.compute)
        for l in range(L):
            a = self.args(l)
            tel = self.telemetry[l]
            mira.mira_moe_route(self.shape, a, self.compute)
            tgt = l + 2
            predicting = mode == "predict" and tgt < L
            if predicting:
                # the head for layer l+2 needs only layer l's input and routing:
                # it runs on the side stream while layer l's experts run
                routed = torch.cuda.Event()
                routed.record(self.compute)
                self.side.wait_event(routed)
                self._predict(l)
            self.counts_h.copy_(self.counts, non_blocking=True)
            self.compute.synchronize()
            cnt = [int(self.counts_h[e]) for e in range(self.E)]
            for e in range(self.E):
                if cnt[e] == 0:
                    continue
                if e in self.hot_slot[l]:
                    slot, tier = self.hot_slot[l][e], "hot"
                    st.hot_hits += 1
                    st.hot_tokens += cnt[e]
                else:
                    slot, tier = self._staged(l, e), "stage"
                    if slot >= 0:
                        st.stage_hits += 1
                        st.stage_tokens += cnt[e]
                    else:
                        slot, tier = self._stage(l, e, l, True, st, copy_events), "cpu"
                        st.misses += 1
                        st.cpu_tokens += cnt[e]
                self._use(l, e, slot, stall_events)
                tel.record(e, cnt[e], tier)
            tel.advance(self.T)
            mira.mira_moe_experts(self.shape, a, self.compute)
            if on_layer is not None:
                on_layer(l, self.out)
            # the STAGE entries of layer l no longer back its table
            for i in range(self.n_slots):
                if self.role[i] == "stage" and self.held[i] is not None and self.held[i][0] == l:
                    self._unset(l, self.held[i][1])
                    if self.vram_mode == "small":
                        self.held[i], self.ready[i] = None, None
            # prefetch controller: experts of layer l+2
            if tgt < L and mode != "demand":
                if predicting:
                    self.side.synchronize()
                    s = self.scores_h.sum(dim=0)
                    want = sorted(range(self.E), key=lambda e: (-float(s[e]), e))[:stage_per_layer]
                else:  # oracle
                    want = sorted(set(true_idx[tgt].reshape(-1).tolist()))
                for e in want:
                    if e in self.hot_slot[tgt] or self._staged(tgt, e) >= 0:
                        st.prefetch_cached += 1
                    elif self._stage(tgt, e, l + 1, False, st, copy_events) >= 0:
                        st.prefetches += 1
            if self.rebalancer is not None and self.rebalancer.due(tel):
                self._rebalance(l, st, copy_events)
        w1.record(self.compute)
        torch.cuda.synchronize()
        st.wall_ms = w0.elapsed_time(w1)
        st.copy_ms = sum(a.elapsed_time(b) for a, b in copy_events)
        st.stall_ms = sum(a.elapsed_time(b) for a, b in stall_events)
        return st

    def reset_stage(self):
        """Forget every STAGE slot (their table entries back to -1)."""
        torch.cuda.synchronize()
        for i in range(self.n_slots):
            if self.role[i] == "stage" and self.held[i] is not None:
                l, e = self.held[i]
                self._unset(l, e)
                self.held[i], self.ready[i] = None, None
        torch.cuda.synchronize()
