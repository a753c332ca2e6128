"""A stack of MoE layers over a device expert pool with HOT and STAGE slots.

Paper sections IV-C (HOT and STAGE regions of the expert cache), IV-D
(telemetry-driven rebalancing of the HOT set), IV-E (predictive staging of
layer l+2's experts on a copy stream) and IV-F (the staging copies overlap the
compute stream).  The policy runs in the library's native runtime
(mira_stack_*; see include/mira.h for the per-layer rules); this class only
owns the torch tensors the runtime works on (slot pool, slot tables, the
layers' inputs and the call's outputs), registers the CPU-store blobs and
passes each layer's arguments and predictor head.
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
    prefetch_cached: int = 0     # predicted expert already in HOT or STAGE ("prefetch skipped")
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
    cov_hits: int = 0            # Coverage@m numerator and denominator (routed pairs)
    cov_total: int = 0

    def add(self, o: "StepStats"):
        for k in self.__dataclass_fields__:
            setattr(self, k, getattr(self, k) + getattr(o, k))

    @property
    def coverage(self) -> float:
        return self.cov_hits / self.cov_total if self.cov_total else 0.0


@dataclass
class LayerData:
    x: torch.Tensor             # [T][C] activations of the layer (teacher forcing)
    w_router: torch.Tensor      # [E][C]
    bias: torch.Tensor | None   # [E] fp32
    hot: list                   # experts resident in HOT slots at the start
    host: dict = field(default_factory=dict)  # expert -> pinned packed blob (the CPU store)
    pred: object = None         # head scoring layer l+2: (w1, b1, w2, b2) of the MLP head,
                                # or mira.MixtureWeights of a MixtureHead


class ExpertStack:
    """L layers of one MoE shape sharing a slot pool: one HOT slot per resident
    expert of every layer (in layer order), then n_stage STAGE slots.  The
    caller writes each HOT slot's bytes (hot_slot tells where) and fills
    LayerData.host with the CPU store before the first step."""

    def __init__(self, shape: mira.MoEShape, tokens: int, layers: list, stride: int,
                 n_stage: int, pred_shape=None, device="cuda",
                 vram_mode: str = "large", rebalancer=None, stage_per_layer: int = 2,
                 lookahead: int = 2):
        if vram_mode not in ("small", "large"):
            raise ValueError("vram_mode must be 'small' or 'large'")
        self.shape, self.T, self.layers, self.stride = shape, tokens, layers, stride
        self.E = shape.n_experts
        self.G = shape.n_experts + shape.n_shared
        self.device = device
        self.n_hot = sum(len(ld.hot) for ld in layers)
        self.n_stage = n_stage
        self.n_slots = self.n_hot + n_stage
        self.vram_mode, self.rebalancer = vram_mode, rebalancer
        self.stage_per_layer = stage_per_layer
        self.pool = torch.zeros(max(1, self.n_slots) * stride, dtype=torch.uint8, device=device)
        self.tables = torch.full((len(layers), self.G), -1, dtype=torch.int32, device=device)
        rb = dict(rb_interval=0)
        if rebalancer is not None:
            c = rebalancer.cfg
            rb = dict(rb_interval=c.interval, rb_max_swaps=c.max_swaps, rb_probation=c.probation,
                      rb_margin=c.margin, rb_miss_weight=c.miss_weight)
        self.cfg = mira.stack_config(len(layers), self.n_hot, n_stage, tokens, stride,
                                     mira.MIRA_VRAM_SMALL if vram_mode == "small" else mira.MIRA_VRAM_LARGE,
                                     lookahead, stage_per_layer, **rb)
        self.compute = torch.cuda.current_stream(device)
        self.handle = mira.mira_stack_create(self.cfg, shape, self.pool, self.tables, self.compute)
        s = 0
        for l, ld in enumerate(layers):
            for e in ld.hot:
                mira.mira_stack_set_hot(self.handle, l, e, s, copy=False)
                s += 1
        self.ws = torch.empty(mira.mira_workspace_bytes(shape, tokens), dtype=torch.uint8, device=device)
        self.out = torch.empty((tokens, shape.hidden), dtype=torch.float32, device=device)
        self.idx = torch.empty((tokens, shape.top_k), dtype=torch.int32, device=device)
        self.counts = torch.zeros((self.G,), dtype=torch.int32, device=device)
        self.status = torch.zeros((1,), dtype=torch.int32, device=device)
        self.pred_shape, self.mixture, self.logits = None, False, None
        self._registered = {}
        self.set_predictor(pred_shape)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h:
            try:
                mira.mira_stack_destroy(h)
            except Exception:  # interpreter shutdown
                pass
            self.handle = None

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

    def args(self, l: int) -> mira.MoEArgs:
        ld = self.layers[l]
        return mira.MoEArgs(x=ld.x, n_tokens=self.T, n_slots=self.n_slots, w_router=ld.w_router,
                            router_bias=ld.bias, slot_table=self.tables[l], slot_pool=self.pool,
                            slot_stride=self.stride, out=self.out, topk_idx=self.idx,
                            logits=self.logits, expert_counts=self.counts, status=self.status, workspace=self.ws,
                            workspace_bytes=self.ws.numel())

    @property
    def hot_slot(self) -> list:
        """Per layer: {expert: HOT slot}."""
        out = []
        for l in range(len(self.layers)):
            m = {}
            for e in range(self.G):
                s = mira.mira_stack_find(self.handle, l, e, 0)
                if s >= 0:
                    m[e] = s
            out.append(m)
        return out

    def hot_set(self, l: int) -> set:
        return {e for e in range(self.G) if mira.mira_stack_find(self.handle, l, e, 0) >= 0}

    def staged(self, l: int, e: int) -> int:
        return mira.mira_stack_find(self.handle, l, e, 1)

    def _register_host(self):
        for l, ld in enumerate(self.layers):
            for e, blob in ld.host.items():
                if self._registered.get((l, e)) is not blob:
                    mira.mira_stack_set_host(self.handle, l, e, blob, blob.numel())
                    self._registered[l, e] = blob

    def _head(self, l: int, mode: str, true_idx):
        tgt = l + self.cfg.lookahead
        if tgt >= len(self.layers) or mode == "demand":
            return None
        if mode == "oracle":
            return mira.stack_head(mira.MIRA_HEAD_GIVEN, given=sorted(set(true_idx[tgt].reshape(-1).tolist())))
        if mode != "predict":
            raise ValueError(f"unknown mode {mode!r}")
        ld = self.layers[l]
        if ld.pred is None:
            return None
        if self.mixture:
            return mira.stack_head(mira.MIRA_HEAD_MIXTURE, mix_shape=self.pred_shape, mix=ld.pred,
                                   workspace=self.pws, workspace_bytes=self.pws.numel())
        w1, b1, w2, b2 = ld.pred
        return mira.stack_head(mira.MIRA_HEAD_MLP, mlp_shape=self.pred_shape, w1=w1, b1=b1, w2=w2, b2=b2,
                               workspace=self.pws, workspace_bytes=self.pws.numel())

    # ---- one decode step through every layer ------------------------------
    def step(self, mode: str = "predict", true_idx=None, on_layer=None) -> StepStats:
        """One decode step through every layer.  mode: "predict" (the layers'
        heads pick layer l+2's experts), "oracle" (stage every expert layer
        l+2 selects, from true_idx, its routing on an earlier pass; an upper
        bound) or "demand" (no prefetch).  on_layer(l, out), if given, is
        called after layer l's experts are queued (out is reused by the next
        layer, so copy it on the compute stream)."""
        self._register_host()
        mira.mira_stack_begin_step(self.handle)
        try:
            for l in range(len(self.layers)):
                mira.mira_stack_layer(self.handle, l, self.args(l), self._head(l, mode, true_idx))
                if on_layer is not None:
                    on_layer(l, self.out)
        finally:
            st = mira.mira_stack_end_step(self.handle)
        return StepStats(**st)

    def events(self) -> list:
        """The runtime's event log since the last read: (kind, layer, target, expert, slot)."""
        return mira.mira_stack_read_events(self.handle)

    def reset_stage(self):
        """Forget every STAGE slot."""
        mira.mira_stack_reset_stage(self.handle)
