"""A stack of MoE layers over a device expert pool with HOT and STAGE slots.

Paper sections IV-C (HOT and STAGE regions of the expert cache), IV-E
(predictive staging of layer l+2's experts on a copy stream) and IV-F (the
staging copies overlap the compute stream).  This module is the host-side
bookkeeping of a decode step through L layers; every byte still moves through
the library: mira_moe_route / mira_moe_experts run a layer, mira_predict
scores layer l+2's experts, mira_stage_expert copies a packed expert from
pinned host memory into a slot on the copy stream, and mira_set_slot updates a
layer's slot table in stream order.

Policy, per layer l of a step:
  1. route layer l; read which experts its tokens selected;
  2. every selected expert is served from its HOT slot, from a STAGE slot
     filled earlier (the compute stream waits for that copy), or by a demand
     copy into a free STAGE slot (a miss);
  3. run the experts of layer l;
  4. choose experts of layer l+2 and copy them into free STAGE slots ahead of
     time: mode "predict" stages the `stage_per_layer` best-scored non-HOT
     experts of the predictor head, mode "oracle" stages every non-HOT expert
     layer l+2 will select (an upper bound), mode "demand" stages nothing.
STAGE slots whose layer has passed are free again (drop when passed); when no
slot is free a prefetch is skipped and a miss waits for the oldest slot of a
passed layer.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

from . import _binding as mira


@dataclass
class StepStats:
    hot_hits: int = 0
    stage_hits: int = 0
    misses: int = 0
    prefetches: int = 0
    prefetch_skipped: int = 0
    h2d_bytes: int = 0
    copy_ms: float = 0.0      # summed durations of the staging copies (copy stream)
    stall_ms: float = 0.0     # time the compute stream waited for copies
    wall_ms: float = 0.0

    def add(self, o: "StepStats"):
        for k in self.__dataclass_fields__:
            setattr(self, k, getattr(self, k) + getattr(o, k))


@dataclass
class LayerData:
    x: torch.Tensor             # [T][C] activations of the layer (teacher forcing)
    w_router: torch.Tensor      # [E][C]
    bias: torch.Tensor | None   # [E] fp32
    hot: list                   # experts resident in HOT slots
    host: dict = field(default_factory=dict)  # expert -> pinned packed blob (non-HOT experts)
    pred: tuple | None = None   # (w1, b1, w2, b2) of the head scoring layer l+2


class ExpertStack:
    """L layers of one MoE shape sharing a slot pool: one HOT slot per resident
    expert of every layer, then n_stage STAGE slots."""

    def __init__(self, shape: mira.MoEShape, tokens: int, layers: list, stride: int,
                 n_stage: int, pred_shape: mira.PredShape | None = None, device="cuda"):
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
        self.pool = torch.zeros(self.n_slots * stride, dtype=torch.uint8, device=device)
        self.tables = torch.full((len(layers), self.E), -1, dtype=torch.int32, device=device)
        self.hot_slot = []
        s = 0
        for l, ld in enumerate(layers):
            m = {}
            for e in ld.hot:
                m[e] = s
                s += 1
            self.hot_slot.append(m)
            for e, slot in m.items():
                self.tables[l, e] = slot
        self.ws = torch.empty(mira.mira_workspace_bytes(shape, tokens), dtype=torch.uint8, device=device)
        self.out = torch.empty((tokens, shape.hidden), dtype=torch.float32, device=device)
        self.idx = torch.empty((tokens, shape.top_k), dtype=torch.int32, device=device)
        self.counts = torch.zeros((self.E + shape.n_shared,), dtype=torch.int32, device=device)
        self.counts_h = torch.zeros_like(self.counts, device="cpu").pin_memory()
        self.status = torch.zeros((1,), dtype=torch.int32, device=device)
        self.pred_shape = pred_shape
        if pred_shape is not None:
            self.pws = torch.empty(mira.mira_predict_workspace_bytes(pred_shape, tokens), dtype=torch.uint8,
                                   device=device)
            self.scores = torch.empty((tokens // pred_shape.group, pred_shape.n_out), dtype=torch.float32,
                                      device=device)
            self.scores_h = torch.zeros(self.scores.shape, dtype=torch.float32).pin_memory()
        self.compute = torch.cuda.current_stream(device)
        self.copy = torch.cuda.Stream(device)  # default priority
        # STAGE slot state: (layer, expert) held, event of its copy
        self.stage_of = [None] * n_stage
        self.stage_ev = [None] * n_stage
        self.stage_age = [0] * n_stage
        self.clock = 0

    def hot_slot_of(self, l: int, e: int) -> int:
        return self.hot_slot[l][e]

    def args(self, l: int) -> mira.MoEArgs:
        ld = self.layers[l]
        return mira.MoEArgs(x=ld.x, n_tokens=self.T, n_slots=self.n_slots, w_router=ld.w_router,
                            router_bias=ld.bias, slot_table=self.tables[l], slot_pool=self.pool,
                            slot_stride=self.stride, out=self.out, topk_idx=self.idx,
                            expert_counts=self.counts, status=self.status, workspace=self.ws,
                            workspace_bytes=self.ws.numel())

    # ---- STAGE slots ------------------------------------------------------
    def _find(self, l, e):
        for i, held in enumerate(self.stage_of):
            if held == (l, e):
                return i
        return -1

    def _free_slot(self, cur_layer, for_demand):
        """A STAGE slot for a copy made while layer cur_layer is current: a free
        slot, else the oldest slot of a passed layer; a demand copy may also
        take the oldest prefetch for a later layer (that prefetch is lost).
        Slots holding the current layer's experts are never taken."""
        cands = [i for i, h in enumerate(self.stage_of) if h is None or h[0] < cur_layer]
        if not cands and for_demand:
            cands = [i for i, h in enumerate(self.stage_of) if h[0] > cur_layer]
        if not cands:
            return -1
        free = [i for i in cands if self.stage_of[i] is None]
        return free[0] if free else min(cands, key=lambda i: self.stage_age[i])

    def _stage(self, l, e, cur_layer, for_demand, st: StepStats, copy_events):
        i = self._free_slot(cur_layer, for_demand)
        if i < 0:
            if for_demand:  # cannot happen with n_stage >= experts per layer outside HOT
                raise RuntimeError("no STAGE slot free for a demand copy")
            st.prefetch_skipped += 1
            return -1
        # (a slot's table entry is set only while its layer runs, so an evicted
        # slot backs no table entry) the copy must not overwrite the slot
        # before the kernels already queued on the compute stream are done with it
        ready = torch.cuda.Event()
        ready.record(self.compute)
        self.copy.wait_event(ready)
        t0, t1, done = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
                        torch.cuda.Event())
        t0.record(self.copy)
        blob = self.layers[l].host[e]
        mira.mira_stage_expert(self.pool, self.stride, self.n_hot + i, blob, blob.numel(), self.copy, None)
        t1.record(self.copy)
        done.record(self.copy)
        copy_events.append((t0, t1))
        st.h2d_bytes += blob.numel()
        self.stage_of[i] = (l, e)
        self.stage_ev[i] = done
        self.clock += 1
        self.stage_age[i] = self.clock
        return i

    # ---- one decode step through every layer ------------------------------
    def step(self, mode: str = "predict", stage_per_layer: int = 2, true_idx=None,
             on_layer=None) -> StepStats:
        """One decode step through every layer.  true_idx[l] (the routing of
        layer l) is needed by mode "oracle"; on_layer(l, out), if given, is
        called after layer l's experts are queued (out is reused by the next
        layer, so copy it on the compute stream)."""
        st = StepStats()
        L = len(self.layers)
        copy_events, stall_events = [], []
        w0, w1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        w0.record(self.compute)
        for l in range(L):
            a = self.args(l)
            mira.mira_moe_route(self.shape, a, self.compute)
            self.counts_h.copy_(self.counts, non_blocking=True)
            self.compute.synchronize()
            sel = [e for e in range(self.E) if int(self.counts_h[e]) > 0]
            for e in sel:
                if e in self.hot_slot[l]:
                    st.hot_hits += 1
                    continue
                i = self._find(l, e)
                if i >= 0:
                    st.stage_hits += 1
                else:
                    st.misses += 1
                    i = self._stage(l, e, l, True, st, copy_events)
                b, c = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                b.record(self.compute)
                self.compute.wait_event(self.stage_ev[i])
                c.record(self.compute)
                stall_events.append((b, c))
                mira.mira_set_slot(self.tables[l], e, self.n_hot + i, self.compute)
            mira.mira_moe_experts(self.shape, a, self.compute)
            if on_layer is not None:
                on_layer(l, self.out)
            # lookahead: experts of layer l+2
            tgt = l + 2
            if tgt < L and mode != "demand":
                if mode == "predict":
                    w1p, b1p, w2p, b2p = self.layers[l].pred
                    mira.mira_predict(self.pred_shape, self.layers[l].x, self.T, w1p, b1p, w2p, b2p,
                                      self.scores, self.pws, self.pws.numel(), self.compute)
                    self.scores_h.copy_(self.scores, non_blocking=True)
                    self.compute.synchronize()
                    s = self.scores_h.sum(dim=0)
                    order = sorted(range(self.E), key=lambda e: (-float(s[e]), e))
                    want = [e for e in order if e not in self.hot_slot[tgt]][:stage_per_layer]
                else:  # oracle
                    want = sorted(e for e in set(true_idx[tgt].reshape(-1).tolist())
                                  if e not in self.hot_slot[tgt])
                for e in want:
                    if self._find(tgt, e) < 0:
                        if self._stage(tgt, e, l + 1, False, st, copy_events) >= 0:
                            st.prefetches += 1
            # a STAGE slot of layer l no longer backs its table entry once the layer passed
            for i, held in enumerate(self.stage_of):
                if held is not None and held[0] == l:
                    mira.mira_set_slot(self.tables[l], held[1], -1, self.compute)
        w1.record(self.compute)
        torch.cuda.synchronize()
        st.wall_ms = w0.elapsed_time(w1)
        st.copy_ms = sum(a.elapsed_time(b) for a, b in copy_events)
        st.stall_ms = sum(a.elapsed_time(b) for a, b in stall_events)
        return st

    def reset_stage(self):
        """Forget every STAGE slot (their table entries back to -1)."""
        torch.cuda.synchronize()
        for i, held in enumerate(self.stage_of):
            if held is not None:
                self.tables[held[0], held[1]] = -1
        self.stage_of = [None] * self.n_stage
        self.stage_ev = [None] * self.n_stage
        self.stage_age = [0] * self.n_stage
        torch.cuda.synchronize()
