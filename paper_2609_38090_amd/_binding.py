"""ctypes binding of libmira.so: argument marshalling only."""
from __future__ import annotations

import ctypes
import os
import threading
from dataclasses import dataclass, field, fields
from typing import Any, Optional

_PKG = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libmira.so"

MIRA_F32 = 0
MIRA_BF16 = 1
MIRA_FLAG_SOFTMAX_ALL = 0x1
MIRA_FLAG_FORCE_DECODE = 0x2
MIRA_FLAG_FORCE_PREFILL = 0x4
MIRA_FLAG_INT4 = 0x8
MIRA_DECODE_MAX_TOKENS = 16
MIRA_MAX_EXPERTS = 256
MIRA_MAX_TOPK = 16
MIRA_NOALLOC_SCRATCH_BYTES = 16 << 20
MIRA_VRAM_LARGE, MIRA_VRAM_SMALL = 0, 1
MIRA_HEAD_NONE, MIRA_HEAD_MLP, MIRA_HEAD_MIXTURE, MIRA_HEAD_GIVEN = 0, 1, 2, 3
MIRA_STACK_EVENTS = ("hot_hit", "stage_hit", "demand", "predicted", "prefetch", "prefetch_cached",
                     "prefetch_declined", "prefetch_dropped", "swap_relabel", "swap_copy", "evict")


class MiraError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"mira error {code}: {msg}")
        self.code = code


class _Shape(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("ffn", ctypes.c_int32), ("n_experts", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("n_shared", ctypes.c_int32), ("act_dtype", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("reserved", ctypes.c_int32)]


class _Args(ctypes.Structure):
    _fields_ = [("x", ctypes.c_void_p), ("n_tokens", ctypes.c_int32), ("n_slots", ctypes.c_int32),
                ("w_router", ctypes.c_void_p), ("router_bias", ctypes.c_void_p),
                ("slot_table", ctypes.c_void_p), ("slot_pool", ctypes.c_void_p),
                ("slot_stride", ctypes.c_uint64), ("out", ctypes.c_void_p),
                ("topk_idx", ctypes.c_void_p), ("topk_weight", ctypes.c_void_p),
                ("logits", ctypes.c_void_p), ("expert_counts", ctypes.c_void_p),
                ("status", ctypes.c_void_p), ("expert_offsets", ctypes.c_void_p),
                ("pair_order", ctypes.c_void_p), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_uint64)]


class _PredShape(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("pred_hidden", ctypes.c_int32), ("n_out", ctypes.c_int32),
                ("group", ctypes.c_int32), ("act_dtype", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class _MixShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("hidden", "n_src", "top_k", "hist_top", "act_hidden",
                                              "hist_hidden", "n_out", "group", "act_dtype", "reserved")]


_MIX_PTRS = ("wah", "wal", "ba1", "wa2", "ba2", "whq", "whu", "bh1", "wh2", "bh2", "gh", "gl", "gq", "gu")


class _MixWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in _MIX_PTRS] + [("bg", ctypes.c_float),
                                                             ("reserved", ctypes.c_int32)]


@dataclass
class MoEShape:
    """mira_shape: C (hidden), R (ffn), E, k, S, activation dtype and flags."""
    hidden: int
    ffn: int
    n_experts: int
    top_k: int
    n_shared: int = 0
    act_dtype: int = MIRA_BF16
    flags: int = 0

    def _c(self) -> _Shape:
        return _Shape(self.hidden, self.ffn, self.n_experts, self.top_k, self.n_shared,
                      self.act_dtype, self.flags, 0)


@dataclass
class PredShape:
    """mira_pred_shape: C, P (MLP width), scored experts, pooled rows per evaluation."""
    hidden: int
    pred_hidden: int
    n_out: int
    group: int
    act_dtype: int = MIRA_BF16

    def _c(self) -> _PredShape:
        return _PredShape(self.hidden, self.pred_hidden, self.n_out, self.group, self.act_dtype, 0)


@dataclass
class MixtureShape:
    """mira_mixture_shape: C, source experts E, k, top-m, head widths, scored experts, group."""
    hidden: int
    n_src: int
    top_k: int
    hist_top: int
    act_hidden: int
    hist_hidden: int
    n_out: int
    group: int
    act_dtype: int = MIRA_BF16

    def _c(self) -> _MixShape:
        return _MixShape(self.hidden, self.n_src, self.top_k, self.hist_top, self.act_hidden,
                         self.hist_hidden, self.n_out, self.group, self.act_dtype, 0)


@dataclass
class MixtureWeights:
    """mira_mixture_weights.  Tensor fields take torch tensors, integer addresses or None."""
    wah: Any = None
    wal: Any = None
    ba1: Any = None
    wa2: Any = None
    ba2: Any = None
    whq: Any = None
    whu: Any = None
    bh1: Any = None
    wh2: Any = None
    bh2: Any = None
    gh: Any = None
    gl: Any = None
    gq: Any = None
    gu: Any = None
    bg: float = 0.0

    def _c(self) -> _MixWeights:
        return _MixWeights(**{n: _ptr(getattr(self, n)) for n in _MIX_PTRS}, bg=float(self.bg), reserved=0)


@dataclass
class MoEArgs:
    """mira_moe_args.  Pointer fields take torch tensors, integer addresses or None."""
    x: Any = None
    n_tokens: int = 0
    n_slots: int = 0
    w_router: Any = None
    router_bias: Any = None
    slot_table: Any = None
    slot_pool: Any = None
    slot_stride: int = 0
    out: Any = None
    topk_idx: Any = None
    topk_weight: Any = None
    logits: Any = None
    expert_counts: Any = None
    status: Any = None
    expert_offsets: Any = None
    pair_order: Any = None
    workspace: Any = None
    workspace_bytes: int = 0

    def _c(self) -> _Args:
        vals = {}
        for f in fields(self):
            v = getattr(self, f.name)
            vals[f.name] = v if f.name in ("n_tokens", "n_slots", "slot_stride", "workspace_bytes") else _ptr(v)
        return _Args(**vals)


def _ptr(v) -> Optional[int]:
    if v is None:
        return None
    if isinstance(v, int):
        return v or None
    if hasattr(v, "data_ptr"):
        return v.data_ptr() or None
    raise TypeError(f"cannot take the address of {type(v).__name__}")


def _stream(s) -> Optional[int]:
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream or None
    if isinstance(s, int):
        return s or None
    if hasattr(s, "cuda_stream"):
        return s.cuda_stream or None
    raise TypeError("stream must be a torch stream, an integer hipStream_t or None")


_LIB = None
_LOCK = threading.Lock()


def lib_path() -> str:
    return os.path.join(_PKG, _LIB_NAME)


class _StackConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_hot", ctypes.c_int32), ("n_stage", ctypes.c_int32),
                ("max_tokens", ctypes.c_int32), ("slot_stride", ctypes.c_uint64),
                ("vram_mode", ctypes.c_int32), ("lookahead", ctypes.c_int32),
                ("stage_per_layer", ctypes.c_int32), ("rb_interval", ctypes.c_int32),
                ("rb_max_swaps", ctypes.c_int32), ("rb_probation", ctypes.c_int32),
                ("rb_margin", ctypes.c_int32), ("rb_miss_weight", ctypes.c_float)]


STACK_COUNTERS = ("hot_hits", "stage_hits", "misses", "hot_tokens", "stage_tokens", "cpu_tokens",
                  "prefetches", "prefetch_cached", "prefetch_declined", "swaps", "promote_copies",
                  "h2d_bytes", "cov_hits", "cov_total")


class _StackStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in STACK_COUNTERS] + \
        [("copy_ms", ctypes.c_double), ("stall_ms", ctypes.c_double), ("wall_ms", ctypes.c_double)]


class _StackHead(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("n_given", ctypes.c_int32), ("given", ctypes.c_void_p),
                ("mlp_shape", ctypes.c_void_p), ("w1", ctypes.c_void_p), ("b1", ctypes.c_void_p),
                ("w2", ctypes.c_void_p), ("b2", ctypes.c_void_p), ("mix_shape", ctypes.c_void_p),
                ("mix", ctypes.c_void_p), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_uint64)]


class _StackEvent(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("kind", "layer", "target", "expert", "slot", "reserved")]


def load():
    """Load libmira.so (after torch, so both share torch's HIP runtime)."""
    global _LIB
    with _LOCK:
        if _LIB is not None:
            return _LIB
        path = lib_path()
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run paper_2609_38090_amd.build.build() first")
        import torch  # noqa: F401  (loads the HIP runtime the library binds to)
        lib = ctypes.CDLL(path)
        vp, i32, u32, u64, f32, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32,
                                      ctypes.c_uint64, ctypes.c_float, ctypes.c_size_t)
        sig = {
            "mira_packed_expert_bytes": (sz, [i32, i32]),
            "mira_packed_expert_bytes_int4": (sz, [i32, i32]),
            "mira_workspace_bytes": (sz, [ctypes.POINTER(_Shape), i32]),
            "mira_pack_experts": (ctypes.c_int, [ctypes.POINTER(_Shape), i32, i32, vp, vp, vp, f32, vp,
                                                 u64, i32, vp]),
            "mira_moe_forward": (ctypes.c_int, [ctypes.POINTER(_Shape), ctypes.POINTER(_Args), vp]),
            "mira_moe_forward_noalloc": (ctypes.c_int, [ctypes.POINTER(_Shape), ctypes.POINTER(_Args), vp]),
            "mira_moe_route": (ctypes.c_int, [ctypes.POINTER(_Shape), ctypes.POINTER(_Args), vp]),
            "mira_moe_experts": (ctypes.c_int, [ctypes.POINTER(_Shape), ctypes.POINTER(_Args), vp]),
            "mira_predict_workspace_bytes": (sz, [ctypes.POINTER(_PredShape), i32]),
            "mira_predict": (ctypes.c_int, [ctypes.POINTER(_PredShape), vp, i32, vp, vp, vp, vp, vp, vp,
                                            u64, vp]),
            "mira_mixture_workspace_bytes": (sz, [ctypes.POINTER(_MixShape), i32]),
            "mira_predict_mixture": (ctypes.c_int, [ctypes.POINTER(_MixShape), ctypes.POINTER(_MixWeights),
                                                    vp, vp, vp, i32, vp, vp, vp, u64, vp]),
            "mira_stage_expert": (ctypes.c_int, [vp, u64, i32, vp, u64, vp, vp]),
            "mira_set_slot": (ctypes.c_int, [vp, i32, i32, vp]),
            "mira_stack_create": (ctypes.c_int, [ctypes.POINTER(_StackConfig), ctypes.POINTER(_Shape), vp, vp, vp,
                                                 ctypes.POINTER(vp)]),
            "mira_stack_destroy": (ctypes.c_int, [vp]),
            "mira_stack_set_host": (ctypes.c_int, [vp, i32, i32, vp, u64]),
            "mira_stack_set_hot": (ctypes.c_int, [vp, i32, i32, i32, i32]),
            "mira_stack_begin_step": (ctypes.c_int, [vp]),
            "mira_stack_layer": (ctypes.c_int, [vp, i32, ctypes.POINTER(_Args), ctypes.POINTER(_StackHead)]),
            "mira_stack_end_step": (ctypes.c_int, [vp, ctypes.POINTER(_StackStats)]),
            "mira_stack_reset_stage": (ctypes.c_int, [vp]),
            "mira_stack_find": (i32, [vp, i32, i32, i32]),
            "mira_stack_read_events": (ctypes.c_int, [vp, i32, ctypes.POINTER(_StackEvent), ctypes.POINTER(i32)]),
            "mira_rebalance_plan": (ctypes.c_int, [ctypes.POINTER(_StackConfig), i32, vp, vp, vp, vp, vp, vp, i32,
                                                   vp, vp, ctypes.POINTER(i32)]),
            "mira_last_error": (ctypes.c_char_p, []),
            "mira_version": (ctypes.c_char_p, []),
            "mira_profile_enable": (ctypes.c_int, [i32]),
            "mira_profile_select": (ctypes.c_int, [ctypes.c_char_p]),
            "mira_profile_read": (ctypes.c_int, [i32, ctypes.POINTER(ctypes.c_char_p),
                                                 ctypes.POINTER(i32), ctypes.POINTER(ctypes.c_double),
                                                 ctypes.POINTER(i32)]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        del u32
        _LIB = lib
        return lib


def _check(rc: int):
    if rc != 0:
        raise MiraError(rc, mira_last_error())


# ---- entry points (names of the C ABI) -------------------------------------

def mira_last_error() -> str:
    return load().mira_last_error().decode()


def mira_version() -> str:
    return load().mira_version().decode()


def mira_packed_expert_bytes(hidden: int, ffn: int) -> int:
    return int(load().mira_packed_expert_bytes(hidden, ffn))


def mira_packed_expert_bytes_int4(hidden: int, ffn: int) -> int:
    return int(load().mira_packed_expert_bytes_int4(hidden, ffn))


def mira_workspace_bytes(shape: MoEShape, max_tokens: int) -> int:
    n = int(load().mira_workspace_bytes(ctypes.byref(shape._c()), max_tokens))
    if n == 0:
        raise MiraError(-1, "invalid shape for mira_workspace_bytes")
    return n


def mira_pack_experts(shape: MoEShape, n_experts: int, w_dtype: int, w_gate, w_up, w_down,
                      eps: float, packed, packed_stride: int, on_device: int, stream=None):
    st = _stream(stream) if on_device else None
    _check(load().mira_pack_experts(ctypes.byref(shape._c()), n_experts, w_dtype, _ptr(w_gate),
                                    _ptr(w_up), _ptr(w_down), eps, _ptr(packed), packed_stride,
                                    on_device, st))


def mira_moe_forward(shape: MoEShape, args: MoEArgs, stream=None):
    _check(load().mira_moe_forward(ctypes.byref(shape._c()), ctypes.byref(args._c()), _stream(stream)))


def mira_moe_forward_noalloc(shape: MoEShape, args: MoEArgs, stream=None):
    _check(load().mira_moe_forward_noalloc(ctypes.byref(shape._c()), ctypes.byref(args._c()),
                                           _stream(stream)))


def mira_moe_route(shape: MoEShape, args: MoEArgs, stream=None):
    _check(load().mira_moe_route(ctypes.byref(shape._c()), ctypes.byref(args._c()), _stream(stream)))


def mira_moe_experts(shape: MoEShape, args: MoEArgs, stream=None):
    _check(load().mira_moe_experts(ctypes.byref(shape._c()), ctypes.byref(args._c()), _stream(stream)))


def mira_predict_workspace_bytes(pshape: PredShape, n_tokens: int) -> int:
    return int(load().mira_predict_workspace_bytes(ctypes.byref(pshape._c()), n_tokens))


def mira_predict(pshape: PredShape, x, n_tokens: int, w1, b1, w2, b2, scores, workspace,
                 workspace_bytes: int, stream=None):
    _check(load().mira_predict(ctypes.byref(pshape._c()), _ptr(x), n_tokens, _ptr(w1), _ptr(b1),
                               _ptr(w2), _ptr(b2), _ptr(scores), _ptr(workspace), workspace_bytes,
                               _stream(stream)))


def mira_mixture_workspace_bytes(mshape: MixtureShape, n_tokens: int) -> int:
    return int(load().mira_mixture_workspace_bytes(ctypes.byref(mshape._c()), n_tokens))


def mira_predict_mixture(mshape: MixtureShape, weights: MixtureWeights, x, logits, topk_idx,
                         n_tokens: int, probs, alpha, workspace, workspace_bytes: int, stream=None):
    _check(load().mira_predict_mixture(ctypes.byref(mshape._c()), ctypes.byref(weights._c()), _ptr(x),
                                       _ptr(logits), _ptr(topk_idx), n_tokens, _ptr(probs), _ptr(alpha),
                                       _ptr(workspace), workspace_bytes, _stream(stream)))


def mira_stage_expert(slot_pool, slot_stride: int, slot: int, pinned_src, nbytes: int,
                      copy_stream=None, done_event=None):
    ev = None
    if done_event is not None:
        ev = done_event if isinstance(done_event, int) else done_event.cuda_event
    _check(load().mira_stage_expert(_ptr(slot_pool), slot_stride, slot, _ptr(pinned_src), nbytes,
                                    _stream(copy_stream), ev))


def mira_set_slot(slot_table, expert: int, slot: int, stream=None):
    _check(load().mira_set_slot(_ptr(slot_table), expert, slot, _stream(stream)))


def mira_profile_enable(enable: bool = True):
    _check(load().mira_profile_enable(1 if enable else 0))


def mira_profile_select(kernel_name=None):
    _check(load().mira_profile_select(kernel_name.encode() if kernel_name else None))


def mira_profile_read(max_entries: int = 64):
    """{kernel name: (launches, total ms)} since the last read."""
    lib = load()
    names = (ctypes.c_char_p * max_entries)()
    counts = (ctypes.c_int32 * max_entries)()
    ms = (ctypes.c_double * max_entries)()
    n = ctypes.c_int32(0)
    _check(lib.mira_profile_read(max_entries, names, counts, ms, ctypes.byref(n)))
    return {names[i].decode(): (int(counts[i]), float(ms[i])) for i in range(min(n.value, max_entries))}


# ---- expert cache runtime ---------------------------------------------------

def stack_config(n_layers: int, n_hot: int, n_stage: int, max_tokens: int, slot_stride: int,
                 vram_mode: int = MIRA_VRAM_LARGE, lookahead: int = 2, stage_per_layer: int = 2,
                 rb_interval: int = 0, rb_max_swaps: int = 1, rb_probation: int = 2, rb_margin: int = 1,
                 rb_miss_weight: float = 1.0) -> _StackConfig:
    return _StackConfig(n_layers, n_hot, n_stage, max_tokens, slot_stride, vram_mode, lookahead,
                        stage_per_layer, rb_interval, rb_max_swaps, rb_probation, rb_margin, rb_miss_weight)


def mira_stack_create(cfg: _StackConfig, shape: MoEShape, slot_pool, slot_tables, compute=None) -> int:
    h = ctypes.c_void_p(0)
    _check(load().mira_stack_create(ctypes.byref(cfg), ctypes.byref(shape._c()), _ptr(slot_pool),
                                    _ptr(slot_tables), _stream(compute), ctypes.byref(h)))
    return h.value


def mira_stack_destroy(st: int):
    _check(load().mira_stack_destroy(st))


def mira_stack_set_host(st: int, layer: int, expert: int, pinned, nbytes: int):
    _check(load().mira_stack_set_host(st, layer, expert, _ptr(pinned), nbytes))


def mira_stack_set_hot(st: int, layer: int, expert: int, slot: int, copy: bool = False):
    _check(load().mira_stack_set_hot(st, layer, expert, slot, 1 if copy else 0))


def mira_stack_begin_step(st: int):
    _check(load().mira_stack_begin_step(st))


def stack_head(kind: int = MIRA_HEAD_NONE, given=None, mlp_shape: "PredShape | None" = None, w1=None,
               b1=None, w2=None, b2=None, mix_shape: "MixtureShape | None" = None,
               mix: "MixtureWeights | None" = None, workspace=None, workspace_bytes: int = 0):
    """A mira_stack_head; the returned tuple keeps the structures it points to alive."""
    keep = []
    h = _StackHead(kind=kind, workspace=_ptr(workspace), workspace_bytes=workspace_bytes)
    if given is not None:
        arr = (ctypes.c_int32 * max(1, len(given)))(*[int(e) for e in given])
        keep.append(arr)
        h.n_given, h.given = len(given), ctypes.cast(arr, ctypes.c_void_p).value
    if mlp_shape is not None:
        ps = mlp_shape._c()
        keep.append(ps)
        h.mlp_shape = ctypes.addressof(ps)
        h.w1, h.b1, h.w2, h.b2 = _ptr(w1), _ptr(b1), _ptr(w2), _ptr(b2)
    if mix_shape is not None:
        ms, mw = mix_shape._c(), mix._c()
        keep += [ms, mw]
        h.mix_shape, h.mix = ctypes.addressof(ms), ctypes.addressof(mw)
    return h, keep


def mira_stack_layer(st: int, layer: int, args: MoEArgs, head=None):
    hp = None if head is None else ctypes.byref(head[0])
    _check(load().mira_stack_layer(st, layer, ctypes.byref(args._c()), hp))


def mira_stack_end_step(st: int) -> dict:
    s = _StackStats()
    _check(load().mira_stack_end_step(st, ctypes.byref(s)))
    return {n: getattr(s, n) for n, _ in _StackStats._fields_}


def mira_stack_reset_stage(st: int):
    _check(load().mira_stack_reset_stage(st))


def mira_stack_find(st: int, layer: int, expert: int, role: int) -> int:
    return int(load().mira_stack_find(st, layer, expert, role))


def mira_stack_read_events(st: int, max_events: int = 65536) -> list:
    """[(kind name, layer, target, expert, slot)] logged since the last read, oldest first."""
    buf = (_StackEvent * max_events)()
    n = ctypes.c_int32(0)
    _check(load().mira_stack_read_events(st, max_events, buf, ctypes.byref(n)))
    return [(MIRA_STACK_EVENTS[buf[i].kind], buf[i].layer, buf[i].target, buf[i].expert, buf[i].slot)
            for i in range(n.value)]


def mira_rebalance_plan(cfg: _StackConfig, routed, cpu, last_use, history, hist_len, is_hot,
                        max_swaps_out: int = 64):
    """Swaps [(evict, promote)] of one rebalancing pass; array arguments are
    numpy arrays (int32 routed/cpu/hist_len [n], int64 last_use [n], int32
    history [n][8], uint8 is_hot [n])."""
    import numpy as np
    n = len(routed)
    arrs = [np.ascontiguousarray(a, dtype=t) for a, t in ((routed, np.int32), (cpu, np.int32),
                                                         (last_use, np.int64), (history, np.int32),
                                                         (hist_len, np.int32), (is_hot, np.uint8))]
    ev = np.zeros(max_swaps_out, np.int32)
    pr = np.zeros(max_swaps_out, np.int32)
    k = ctypes.c_int32(0)
    _check(load().mira_rebalance_plan(ctypes.byref(cfg), n, *[a.ctypes.data for a in arrs], max_swaps_out,
                                      ev.ctypes.data, pr.ctypes.data, ctypes.byref(k)))
    return [(int(ev[i]), int(pr[i])) for i in range(k.value)]
