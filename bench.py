"""Benchmark of the Mira MoE expert step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

A step is one MoE layer call (router, top-k, permutation, expert FFN over
packed experts, combine) on one batch of the workload.  The beam workload's
step is one decode step of its 8 beams through all 32 layers of the stack,
with 4 of 8 experts per layer resident (HOT slots), the others copied from
pinned host memory into STAGE slots ahead of time (predictor head for layer
l+2, or the true experts as an upper bound) or on demand.  Inputs are seeded synthetic tensors of
the workload's shapes, resident in HBM before timing starts.  Weights are
rotated over several packed copies of the layer so every call streams cold
expert bytes (more than 1 GB between reuses, above the 256 MB Infinity Cache).

Prints one JSON line with the throughput (tokens/s), the roofline of the
dominant kernel (timed with HIP events on its stream inside the timed
region) and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/s (decode+prefill); HBM GB/s on packed experts vs peak"
# The paper's end-to-end speedups over its comparison systems, on its own
# hardware: context for the reader, not a figure this bench measures.
PAPER_CONTEXT = {
    "note": "the paper's end-to-end speedups over other systems on its own GPUs; context only, "
            "not comparable with this line",
    "throughput_vs_moe_infinity": {"speedup": 5.71, "gpu": "RTX A5000 24 GB"},
    "ttft_vs_fiddler": {"speedup": 11.71, "gpu": "RTX 6000 Ada 48 GB"},
    "beam_search_vs_fiddler": {"speedup": 3.84, "gpu": "not stated"},
}
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
COLD_BYTES = 1 << 30
PROF_EVERY = 8  # steps timed with events: one layer-copy rotation in every 8

# HBM bytes per launch of the dominant kernels, from two rocprofv3 --pmc runs
# (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch, averaged) on this bench's
# workload, each scaled by what the same counter reads for a plain 1 GiB
# device copy (bench.py --copy-bytes 1073741824 reads FETCH_SIZE 524302 KiB
# and WRITE_SIZE 1048576 KiB: scale 2.0 and 1.0).  An entry holds only for
# the kernel code it was measured on (hash of the kernel file and the two
# shared headers with comments and spacing dropped); otherwise the bench
# reports traffic as null.
FETCH_SCALE, WRITE_SCALE = 2.0, 1.0
TRAFFIC = {
    ("decode_gateup", "mixtral_decode"): dict(sources=("decode.hip", "decode_dev.h", "int4_format.h"),
                                               sha="2b2b8f93748da802", fetch_kib=114834.8, write_kib=110.3),
    ("decode_gateup", "mixtral_decode_int4"): dict(sources=("decode.hip", "decode_dev.h", "int4_format.h"),
                                                    sha="2b2b8f93748da802", fetch_kib=61622.0, write_kib=110.1),
    # the beam stack's decode_gateup: the mean over all its launches (32
    # layers, 5.38 selected experts per layer on average)
    ("decode_gateup", "beam_stack"): dict(sources=("decode.hip", "decode_dev.h", "int4_format.h"),
                                          sha="2b2b8f93748da802", fetch_kib=308765.0, write_kib=560.3),
    ("prefill_gateup", "mixtral_prefill"): dict(sources=("prefill.hip",), sha="8d87e7443ab4d714",
                                                 fetch_kib=600413.4, write_kib=38203.4),
    ("prefill_gateup", "fine_grained"): dict(sources=("prefill.hip",), sha="8d87e7443ab4d714",
                                              fetch_kib=290638.8, write_kib=57853.3),
}


def strip_comments(text):
    """C/C++ source without its comments and blank space, so that only code
    changes alter a source hash (string literals are kept as they are)."""
    import re
    pat = re.compile(r'//[^\n]*|/\*.*?\*/|"(?:\\.|[^"\\])*"', re.S)
    code = pat.sub(lambda m: m.group(0) if m.group(0).startswith('"') else " ", text)
    return " ".join(code.split())


def source_hash(sources):
    """Hash of the code (comments and spacing dropped) of the kernel sources
    and the two shared headers."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2609_38090_amd", "csrc")
    h = hashlib.sha256()
    for f in tuple(sources) + ("device_util.h", "mira_internal.h"):
        with open(os.path.join(csrc, f), encoding="utf-8") as fh:
            h.update(strip_comments(fh.read()).encode())
    return h.hexdigest()[:16]


def traffic_bytes(kernel, workload):
    """Counter-measured HBM bytes per launch, or None if not measured on these sources."""
    ent = TRAFFIC.get((kernel, workload))
    if ent is None or ent["sha"] is None or source_hash(ent["sources"]) != ent["sha"]:
        return None
    return int((ent["fetch_kib"] * FETCH_SCALE + ent["write_kib"] * WRITE_SCALE) * 1024)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default=None,
                   choices=["tiny", "mixtral_decode", "mixtral_prefill", "fine_grained", "beam_stack"],
                   help="one workload alone; by default mixtral_decode is the headline line and the "
                        "prefill layers and the beam stack are measured after it (key 'workloads')")
    p.add_argument("--format", default="int8", choices=["int8", "int4"],
                   help="expert format: the paper's shared-scale INT8, or the INT4 variant "
                        "(group-64 fp16 scales; decode workloads only)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-profile", action="store_true", help="skip the per-kernel HIP-event timing")
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU oracle sample")
    p.add_argument("--extra-cpu-seconds", type=float, default=6.0,
                   help="budget per oracle leg of the workloads measured after the headline one")
    p.add_argument("--layers", type=int, default=0, help="layers of the beam stack (0 = all)")
    p.add_argument("--stage-slots", type=int, default=8, help="STAGE slots of the beam stack")
    p.add_argument("--drift-steps", type=int, default=36,
                   help="beam stack: steps of the drifting-popularity HOT rebalancing run (0 = skip)")
    p.add_argument("--source-hash", action="store_true",
                   help="print the source hashes the traffic table is keyed on and exit")
    p.add_argument("--scale-bench", action="store_true",
                   help="instead of the MoE step, time staging only the scale metadata of experts: "
                        "one shared scale vector per expert against three per-matrix vectors")
    p.add_argument("--copy-bytes", type=int, default=0,
                   help="instead of the MoE step, time a plain device-to-device copy of this many "
                        "bytes (the reference kernel for scaling the FETCH_SIZE/WRITE_SIZE counters)")
    return p.parse_args()


def copy_reference(nbytes, steps):
    """Plain device copy of known size, for calibrating the HBM byte counters."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / steps
    print(json.dumps({"copy_bytes": nbytes, "steps": steps, "ms_per_copy": round(dt * 1e3, 4),
                      "gbs_read_plus_write": round(2 * nbytes / dt / 1e9, 1)}), flush=True)
    return 0


# Expert shapes of the scale-only staging microbenchmark: hidden C, expert ffn
# R and the experts of one layer (routed + shared) staged together.
SCALE_SHAPES = {
    "mixtral_8x7b": dict(C=4096, R=14336, experts=8),
    "mixtral_8x22b": dict(C=6144, R=16384, experts=8),
    "deepseek_v2_lite": dict(C=2048, R=1408, experts=66),
}


def scale_bench(reps=200):
    """Staging of scale metadata only (section IV-B): the shared format moves
    one bf16 vector of R scales per expert in one copy; per-matrix per-row
    INT8 moves the gate and up row scales (R each) and the down row scales
    (C) in three copies.  Every copy is a mira_stage_expert call (pinned host
    -> device on one stream); the time of a whole layer's experts is taken
    between two events, median over reps."""
    import torch
    import paper_2609_38090_amd as mira

    mira.load()
    st = torch.cuda.Stream()
    out = {}
    for name, sh in SCALE_SHAPES.items():
        C, R, n = sh["C"], sh["R"], sh["experts"]
        layouts = {"shared": [2 * R], "per_matrix": [2 * R, 2 * R, 2 * C]}
        res = {}
        for kind, sizes in layouts.items():
            src = [torch.ones(n * b, dtype=torch.uint8).pin_memory() for b in sizes]
            dst = [torch.empty(n * b, dtype=torch.uint8, device="cuda") for b in sizes]
            times = []
            for it in range(reps + 10):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(st)
                for e in range(n):
                    for s_, d_, b in zip(src, dst, sizes):
                        mira.mira_stage_expert(d_, b, e, s_[e * b:].data_ptr(), b, st, None)
                e1.record(st)
                e1.synchronize()
                if it >= 10:
                    times.append(e0.elapsed_time(e1) * 1e3)
            times.sort()
            med = times[len(times) // 2]
            res[kind] = dict(copies_per_expert=len(sizes), bytes_per_expert=sum(sizes),
                             us_per_layer=round(med, 2), us_per_expert=round(med / n, 3))
        res["latency_ratio"] = round(res["per_matrix"]["us_per_layer"] / res["shared"]["us_per_layer"], 2)
        res["bytes_ratio"] = round((4 * R + 2 * C) / (2 * R), 2)
        out[name] = dict(hidden=C, ffn=R, experts=n, **res)
    line = {"microbenchmark": "scale-only staging, pinned host -> device", "reps": reps, "shapes": out}
    print(json.dumps(line), flush=True)
    return line


def event_step(i, n_copies):
    """Whether timed step i carries the dominant kernel's events: one rotation
    over the layer copies in every PROF_EVERY (each event pair adds a few
    microseconds to its step), so every copy is sampled equally often."""
    return (i // n_copies) % PROF_EVERY == 0


def expert_stride(cfg, fmt):
    import paper_2609_38090_amd as mira
    return (mira.mira_packed_expert_bytes_int4(cfg.C, cfg.R) if fmt == "int4"
            else mira.mira_packed_expert_bytes(cfg.C, cfg.R))


def format_flag(fmt):
    import paper_2609_38090_amd as mira
    return mira.MIRA_FLAG_INT4 if fmt == "int4" else 0


def build_copies(cfg, n_copies, fmt="int8"):
    """n_copies packed copies of the layer (different seeded weights per copy)."""
    import torch
    import paper_2609_38090_amd as mira
    from mira_inputs import activations, expert_weights, router_bias, router_weights

    stride = expert_stride(cfg, fmt)
    act = mira.MIRA_F32 if cfg.act == "f32" else mira.MIRA_BF16
    pack_shape = mira.MoEShape(cfg.C, cfg.R, 1, 1, flags=format_flag(fmt))
    copies = []
    for l in range(n_copies):
        pool = torch.empty(cfg.G * stride, dtype=torch.uint8, device="cuda")
        for e in range(cfg.G):
            wg, wu, wd = expert_weights(cfg, l, e, "cuda")
            mira.mira_pack_experts(pack_shape, 1, mira.MIRA_F32, wg, wu, wd, 1e-8,
                                   pool[e * stride:], stride, 1)
            del wg, wu, wd
        b = router_bias(cfg, l)
        copies.append(dict(
            pool=pool,
            table=torch.arange(cfg.G, dtype=torch.int32, device="cuda"),
            x=activations(cfg, l, "cuda"),
            wr=router_weights(cfg, l, "cuda"),
            bias=None if b is None else b.cuda(),
        ))
    torch.cuda.synchronize()
    return copies, stride, act


def algorithmic_units(cfg, counts, fmt="int8"):
    """Packed-expert bytes and FLOPs one call must touch, from the routed counts.
    INT8: gate and up (2RC) plus the shared scales (2R bytes) for gate/up, RC
    for down; INT4: per 16 rows x 64 columns, 512 bytes of nibbles and 32 of
    fp16 scales (544 bytes), for gate and up, then for down."""
    active = [g for g in range(cfg.G) if counts[g] > 0]
    pairs = int(sum(counts))
    if fmt == "int4":
        tiles = (cfg.R // 16) * (cfg.C // 64)
        gu_bytes = len(active) * 2 * tiles * 544
        dn_bytes = len(active) * tiles * 544
    else:
        gu_bytes = len(active) * (2 * cfg.R * cfg.C + 2 * cfg.R)
        dn_bytes = len(active) * (cfg.C * cfg.R)
    gu_flops = pairs * 4.0 * cfg.C * cfg.R
    dn_flops = pairs * 2.0 * cfg.C * cfg.R
    return dict(active=len(active), pairs=pairs, gu_bytes=gu_bytes, dn_bytes=dn_bytes,
                gu_flops=gu_flops, dn_flops=dn_flops)


def cpu_baseline(cfg, copy0, budget_s, fmt="int8", legs=(None, 8)):
    """The oracle, as it stands, on a bounded sample of the same workload.

    The sample is the first tokens of layer copy 0 (up to 64, as many as fit
    the budget); the experts it needs are packed beforehand (timed apart).
    The forward over the sample repeats until budget_s is spent, once per
    leg: None = every BLAS thread the process has, n = BLAS limited to n
    threads (8 mirrors the paper's 8-core CPU restriction).  Returns the
    first leg's figures with the others under "legs"."""
    import numpy as np
    import oracle
    from mira_inputs import expert_weights
    from threadpoolctl import threadpool_info, threadpool_limits

    def blas_threads():
        return max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] + [1])

    x = copy0["x"].float().cpu().numpy().astype(np.float64)
    wr = copy0["wr"].float().cpu().numpy().astype(np.float64)
    b = None if copy0["bias"] is None else copy0["bias"].cpu().numpy().astype(np.float64)
    logits = oracle.router_logits(x, wr, b)
    idx = oracle.topk_select(logits, cfg.k)
    pack = oracle.pack_expert_int4 if fmt == "int4" else oracle.pack_expert
    # pack the experts the sample needs (offline step, timed separately)
    t0 = time.perf_counter()
    blobs = {}
    tokens = []
    deadline = time.perf_counter() + budget_s
    for t in range(cfg.T):
        need = [int(e) for e in idx[t] if int(e) not in blobs]
        for e in need:
            wg, wu, wd = (w.cpu().numpy() for w in expert_weights(cfg, 0, e, "cuda"))
            blobs[e] = pack(wg, wu, wd)
        tokens.append(t)
        if time.perf_counter() > deadline or len(tokens) >= 64:
            break
    shared = [pack(*(w.cpu().numpy() for w in expert_weights(cfg, 0, cfg.E + s, "cuda")))
              for s in range(cfg.S)]
    pack_s = time.perf_counter() - t0

    class Blobs:
        def __len__(self):
            return cfg.E

        def __getitem__(self, e):
            return blobs[e]

    def leg(threads):
        with threadpool_limits(limits=threads, user_api="blas"):
            used = blas_threads()
            t1 = time.perf_counter()
            reps = 0
            while True:
                oracle.moe_forward(x, wr, b, Blobs(), cfg.k, cfg.C, cfg.R, shared_blobs=shared,
                                   tokens=tokens, fmt=fmt)
                reps += 1
                if time.perf_counter() - t1 >= budget_s or reps >= 1000:
                    break
            fwd_s = time.perf_counter() - t1
        return dict(value=round(reps * len(tokens) / fwd_s, 4), cores=int(used), reps=reps,
                    seconds=round(fwd_s, 2))

    res = [leg(n) for n in legs]
    first = res[0]
    return {
        "value": first["value"],
        "unit": "tokens/s",
        "cores": first["cores"],
        "kind": "oracle",
        "sample": (f"numpy fp64 oracle forward ({fmt} experts; router, top-k, expert FFN one expert at a "
                   f"time, combine) "
                   f"on the first {len(tokens)} token(s) of layer copy 0 of the same workload; "
                   f"{len(blobs) + len(shared)} experts packed beforehand in {pack_s:.1f} s (not timed); "
                   f"{first['reps']} forward pass(es) over the sample took {first['seconds']:.2f} s; "
                   f"BLAS threads {first['cores']}, "
                   f"host CPUs available {len(os.sched_getaffinity(0))}"),
        "legs": [dict(blas_threads=r["cores"], value=r["value"], reps=r["reps"], seconds=r["seconds"])
                 for r in res],
    }


def build_stack(cfg, n_layers, n_stage, hot=None, bias=None, host_all=False, rebalancer=None,
                fmt="int8"):
    """The beam workload's stack: per layer its seeded input, router, HOT experts
    packed into their device slots and the other experts (all of them if
    host_all, as a rebalancer may evict and later promote any expert) packed
    into pinned host memory, one blob each, plus the predictor head scoring
    layer l+2.  hot(l) and bias(l) override the workload's HOT set and bias;
    fmt picks the expert format ("int8" or the "int4" variant)."""
    import torch
    import paper_2609_38090_amd as mira
    from paper_2609_38090_amd.stack import ExpertStack, LayerData
    from mira_inputs import (activations, expert_weights, predictor_weights, resident_experts,
                             router_bias, router_weights)

    stride = expert_stride(cfg, fmt)
    pack_shape = mira.MoEShape(cfg.C, cfg.R, 1, 1, flags=format_flag(fmt))
    layers = []
    for l in range(n_layers):
        b = router_bias(cfg, l) if bias is None else bias(l)
        pred = tuple(t.cuda() for t in predictor_weights(cfg, l, "cpu")) if l + 2 < n_layers else None
        layers.append(LayerData(x=activations(cfg, l, "cuda"), w_router=router_weights(cfg, l, "cuda"),
                                bias=None if b is None else b.cuda(),
                                hot=resident_experts(cfg, l) if hot is None else hot(l), pred=pred))
    shape = mira.MoEShape(cfg.C, cfg.R, cfg.E, cfg.k, cfg.S, mira.MIRA_BF16, format_flag(fmt))
    ps = mira.PredShape(cfg.C, cfg.pred_hidden, cfg.E, cfg.pred_group, mira.MIRA_BF16)
    stack = ExpertStack(shape, cfg.T, layers, stride, n_stage=n_stage, pred_shape=ps, rebalancer=rebalancer)
    n_host = sum(cfg.E if host_all else cfg.E - len(ld.hot) for ld in layers)
    host = torch.empty(n_host * stride, dtype=torch.uint8, pin_memory=True)
    tmp = torch.empty(stride, dtype=torch.uint8, device="cuda")
    hot_slot = stack.hot_slot
    c = 0
    for l, ld in enumerate(layers):
        for e in range(cfg.E):
            wg, wu, wd = expert_weights(cfg, l, e, "cuda")
            is_hot = e in hot_slot[l]
            mira.mira_pack_experts(pack_shape, 1, mira.MIRA_F32, wg, wu, wd, 1e-8, tmp, stride, 1)
            if is_hot:
                slot = hot_slot[l][e]
                stack.pool[slot * stride:(slot + 1) * stride].copy_(tmp)
            if host_all or not is_hot:
                blob = host[c * stride:(c + 1) * stride]
                blob.copy_(tmp)
                ld.host[e] = blob
                c += 1
            del wg, wu, wd
    torch.cuda.synchronize()
    return stack, stride


def run_drift(cfg, n_layers, steps, period, fmt="int8"):
    """HOT rebalancing on a workload whose expert popularity drifts: every
    `period` steps the Zipf ranks of every layer's router bias change.  The
    same inputs run with a static HOT set (the popular experts of the first
    period) and with the telemetry-driven rebalancer; experts outside HOT are
    copied on demand (no prefetch), so the difference is the HOT hit rate."""
    import torch
    from paper_2609_38090_amd.policy import RebalanceConfig, Rebalancer
    from paper_2609_38090_amd.stack import StepStats
    from mira_inputs import activations, drift_bias, drift_hot

    res = {}
    for name in ("static", "rebalanced"):
        rb = Rebalancer(RebalanceConfig(interval=64, max_swaps=1, probation=2)) if name == "rebalanced" else None
        stack, _ = build_stack(cfg, n_layers, max(cfg.E - cfg.resident, 4) + 2,
                               hot=lambda l: drift_hot(cfg, l, 0, cfg.resident),
                               bias=lambda l: drift_bias(cfg, l, 0), host_all=True, rebalancer=rb,
                               fmt=fmt)
        per_epoch = []
        t0 = time.perf_counter()
        for s in range(steps):
            ep = s // period
            for l, ld in enumerate(stack.layers):
                ld.x.copy_(activations(cfg, l, "cuda", base=1 + s))
                ld.bias.copy_(drift_bias(cfg, l, ep).cuda())
            st = stack.step("demand")
            if s % period == 0:
                per_epoch.append(StepStats())
            per_epoch[-1].add(st)
        el = time.perf_counter() - t0
        eps = []
        for ep, st in enumerate(per_epoch):
            tok = st.hot_tokens + st.stage_tokens + st.cpu_tokens
            eps.append(dict(epoch=ep, hot_token_share=round(st.hot_tokens / max(tok, 1), 3),
                            misses_per_step=round(st.misses / period, 2), swaps=st.swaps,
                            h2d_gb_per_step=round(st.h2d_bytes / period / 1e9, 3),
                            ms_per_step=round(st.wall_ms / period, 2)))
        res[name] = dict(epochs=eps, ms_per_step=round(el * 1e3 / steps, 2))
        del stack
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return dict(layers=n_layers, steps=steps, period=period, rebalance="interval 64 tokens, 1 swap, probation 2",
                **res)


MIX_HIST_HIDDEN = 64  # HistHead width of the beam workload's MixtureHeads (ActHead: the MLP's width)


def mixture_heads(cfg, n_layers):
    """MixtureHead of every layer with a layer l+2 (seeded synthetic weights)."""
    import torch
    import paper_2609_38090_amd as mira
    from mira_inputs import mixture_weights

    shape = mira.MixtureShape(cfg.C, cfg.E, cfg.k, cfg.k, cfg.pred_hidden, MIX_HIST_HIDDEN, cfg.E,
                              cfg.pred_group, mira.MIRA_BF16)
    heads = []
    for l in range(n_layers):
        if l + 2 >= n_layers:
            heads.append(None)
            continue
        W = mixture_weights(cfg, l, cfg.pred_hidden, MIX_HIST_HIDDEN)
        heads.append(mira.MixtureWeights(**{k: v.cuda() for k, v in W.items() if torch.is_tensor(v)},
                                         bg=W["bg"]))
    return shape, heads


def head_bytes(cfg, kind, T):
    """Bytes one predictor call must move: weights, inputs and outputs."""
    C, E, P, n = cfg.C, cfg.E, cfg.pred_hidden, T // cfg.pred_group
    if kind == "predict":
        return 2 * P * C + 4 * P + 2 * E * P + 4 * E + 2 * T * C + 4 * n * E
    Ph = MIX_HIST_HIDDEN
    w = 2 * (P * C + P * E + E * P + 2 * Ph * E + E * Ph + C + 3 * E) + 4 * (P + Ph + 2 * E)
    return w + 2 * T * C + 4 * T * E + 4 * T * cfg.k + 4 * n * (E + 1)


def run_heads(cfg, n_layers, stack, heads_mix, mix_shape, reps=50):
    """Both predictor heads alone: one call per decode step of one layer
    (the beam's 8 tokens, one group), and all layers' calls batched into one.
    Per-call time from the library's event pairs around each call."""
    import torch
    import paper_2609_38090_amd as mira

    ld = stack.layers[0]
    T = cfg.T
    logits = torch.randn((T * n_layers, cfg.E), device="cuda")
    idx = torch.randint(0, cfg.E, (T * n_layers, cfg.k), dtype=torch.int32, device="cuda")
    xb = ld.x.repeat(n_layers, 1)
    ps = mira.PredShape(cfg.C, cfg.pred_hidden, cfg.E, cfg.pred_group, mira.MIRA_BF16)
    w1, b1, w2, b2 = ld.pred
    out = {}
    for tokens in (T, T * n_layers):
        n = tokens // cfg.pred_group
        scores = torch.empty((n, cfg.E), device="cuda")
        pws = torch.empty(max(mira.mira_predict_workspace_bytes(ps, tokens),
                              mira.mira_mixture_workspace_bytes(mix_shape, tokens)), dtype=torch.uint8,
                          device="cuda")
        calls = {
            "predict": lambda: mira.mira_predict(ps, xb, tokens, w1, b1, w2, b2, scores, pws, pws.numel()),
            "mixture": lambda: mira.mira_predict_mixture(mix_shape, heads_mix[0], xb, logits, idx, tokens, scores,
                                                         None, pws, pws.numel()),
        }
        for name, fn in calls.items():
            for _ in range(3):
                fn()
            mira.mira_profile_select(name)
            mira.mira_profile_enable(True)
            mira.mira_profile_read()
            for _ in range(reps):
                fn()
            cnt, ms = mira.mira_profile_read().get(name, (0, 0.0))
            mira.mira_profile_enable(False)
            us = ms / max(cnt, 1) * 1e3
            nbytes = head_bytes(cfg, name, tokens)
            out[f"{name}_T{tokens}"] = dict(us_per_call=round(us, 2), predictions=n, bytes=nbytes,
                                            gbs=round(nbytes / max(us, 1e-9) / 1e3, 1))
    mira.mira_profile_select(None)
    torch.cuda.synchronize()
    return out


def run_stack(args, cfg, summary=False, cpu_s=None):
    """Beam workload: one decode step of the 8 beams through every layer of the
    stack, experts served from HOT slots, STAGE slots filled ahead of time, or
    demand copies; reported per mode of the staging policy.  With summary
    (the default bench run) only the three staging modes of the MLP head are
    timed, over a few steps, and the fields are returned instead of printed."""
    import torch
    import paper_2609_38090_amd as mira
    from paper_2609_38090_amd.stack import StepStats

    mira.load()
    L = args.layers or cfg.layers
    t_build = time.perf_counter()
    fmt = args.format
    stack, stride = build_stack(cfg, L, args.stage_slots, fmt=fmt)
    build_s = time.perf_counter() - t_build
    # the true routing of every layer (the oracle-prefetch mode stages it)
    true_idx, active = [], []
    for l in range(L):
        mira.mira_moe_route(stack.shape, stack.args(l))
        torch.cuda.synchronize()
        true_idx.append(stack.idx.cpu().numpy().copy())
        active.append(len(set(true_idx[-1].reshape(-1).tolist())))
    steps = max(1, min(args.steps, 4 if summary else 8))
    warm = max(1, min(args.warmup, 1 if summary else 2))
    cpu_s = (0 if args.no_cpu_baseline else args.cpu_seconds) if cpu_s is None else cpu_s
    modes = {}
    prof = {}
    for mode in ("predict", "oracle", "demand"):
        stack.reset_stage()
        for _ in range(warm):
            stack.step(mode, true_idx=true_idx)
        if mode == "predict" and not args.no_profile:
            mira.mira_profile_select("decode_gateup")
            mira.mira_profile_enable(True)
            mira.mira_profile_read()
        tot = StepStats()
        walls = []
        t0 = time.perf_counter()
        for _ in range(steps):
            t1 = time.perf_counter()
            tot.add(stack.step(mode, true_idx=true_idx))
            torch.cuda.synchronize()
            walls.append((time.perf_counter() - t1) * 1e6)
        el = (time.perf_counter() - t0) / steps
        if mode == "predict" and not args.no_profile:
            prof = mira.mira_profile_read()
            mira.mira_profile_enable(False)
        per = {k: getattr(tot, k) / steps for k in tot.__dataclass_fields__}
        modes[mode] = dict(
            ms_per_step=round(el * 1e3, 3), tokens_per_s=round(cfg.T / el, 2),
            layer_tokens_per_s=round(cfg.T * L / el, 2),
            hot_hits=per["hot_hits"], stage_hits=per["stage_hits"], misses=per["misses"],
            prefetches=per["prefetches"], prefetch_cached=per["prefetch_cached"],
            prefetch_declined=per["prefetch_declined"],
            h2d_gb_per_step=round(per["h2d_bytes"] / 1e9, 3),
            h2d_gbs_busy=round(per["h2d_bytes"] / max(per["copy_ms"], 1e-9) / 1e6, 1),
            h2d_gbs_wall=round(per["h2d_bytes"] / el / 1e9, 1),
            stall_ms_per_step=round(per["stall_ms"], 3),
            per_step_us=percentiles(walls),
        )
        if tot.cov_total:
            # mass-weighted coverage of the staged picks: the head's top 2 in
            # "predict" mode, every true expert of layer l+2 in "oracle" mode
            modes[mode]["coverage"] = round(tot.coverage, 4)
    if summary:
        return stack_summary(cfg, L, fmt, modes, prof, active, steps, warm, build_s, stack, cpu_s)
    # the same policy with the MixtureHead scoring layer l+2
    mix_shape, heads_mix = mixture_heads(cfg, L)
    mlp_shape, heads_mlp = stack.pred_shape, [ld.pred for ld in stack.layers]
    stack.set_predictor(mix_shape, heads_mix)
    stack.reset_stage()
    for _ in range(warm):
        stack.step("predict")
    tot = StepStats()
    t0 = time.perf_counter()
    for _ in range(steps):
        tot.add(stack.step("predict"))
    torch.cuda.synchronize()
    el = (time.perf_counter() - t0) / steps
    per = {k: getattr(tot, k) / steps for k in tot.__dataclass_fields__}
    modes["predict_mixture"] = dict(
        ms_per_step=round(el * 1e3, 3), tokens_per_s=round(cfg.T / el, 2),
        hot_hits=per["hot_hits"], stage_hits=per["stage_hits"], misses=per["misses"],
        prefetches=per["prefetches"], prefetch_cached=per["prefetch_cached"],
        prefetch_declined=per["prefetch_declined"], h2d_gb_per_step=round(per["h2d_bytes"] / 1e9, 3),
        stall_ms_per_step=round(per["stall_ms"], 3), coverage=round(tot.coverage, 4))
    stack.set_predictor(mlp_shape, heads_mlp)
    heads = run_heads(cfg, L - 2, stack, heads_mix, mix_shape)
    ms = modes["predict"]["ms_per_step"]
    roof = stack_roofline(cfg, L, fmt, prof, active)
    line = {
        "metric": METRIC, "value": modes["predict"]["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1,
        "steps": steps, "warmup": warm, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "i8", "data": "synthetic",
        "config": {"workload": cfg.name, "format": fmt, "tokens": cfg.T, "layers": L, "hidden": cfg.C,
                   "experts": cfg.E, "top_k": cfg.k, "ffn": cfg.R, "resident_per_layer": cfg.resident,
                   "stage_slots": args.stage_slots, "predictor": f"{cfg.C}->{cfg.pred_hidden}->{cfg.E}",
                   "activations": cfg.act, "experts_selected_per_layer": round(sum(active) / L, 2)},
        "staging": modes,
        "predictor_heads": dict(mixture=f"ActHead {cfg.C}+{cfg.E}->{cfg.pred_hidden}->{cfg.E}, "
                                        f"HistHead {2 * cfg.E}->{MIX_HIST_HIDDEN}->{cfg.E}, gate {cfg.C + 3 * cfg.E}->1",
                                **heads),
        "setup_s": round(build_s, 1),
        "kernels_us": {k: round(v[1] / v[0] * 1e3, 2) for k, v in prof.items() if v[0]},
        "roofline": roof,
    }
    if args.drift_steps > 0:
        line["drift"] = run_drift(cfg, min(L, 8), args.drift_steps, max(1, args.drift_steps // 3), fmt)
    if cpu_s > 0:
        ld = stack.layers[0]
        line["cpu_baseline"] = cpu_baseline(cfg, dict(x=ld.x, wr=ld.w_router, bias=ld.bias), cpu_s, fmt)
    print(json.dumps(line), flush=True)
    return 0


def stack_roofline(cfg, L, fmt, prof, active):
    """decode_gateup's HBM roofline in the stack: the algorithmic bytes of the
    average layer's selected experts over the kernel's mean event duration."""
    gu_bytes = sum(algorithmic_units(cfg, [1] * a + [0] * (cfg.G - a), fmt)["gu_bytes"] for a in active) / L
    cnt, tot_ms = prof.get("decode_gateup", (0, 0.0))
    if not cnt:
        return None
    dur = tot_ms / cnt * 1e-3
    achieved = gu_bytes / dur / 1e9
    return {"bound": "hbm", "kernel": "decode_gateup", "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic_bytes("decode_gateup", cfg.name if fmt == "int8" else f"{cfg.name}_int4"),
            "avg_us": round(dur * 1e6, 2), "algorithmic_bytes_per_launch": int(gu_bytes),
            "timed_launches": cnt}


def stack_summary(cfg, L, fmt, modes, prof, active, steps, warm, build_s, stack, cpu_s):
    """The beam stack's fields in the default bench line."""
    import torch
    res = {"value": modes["predict"]["tokens_per_s"], "unit": "tokens/s", "steps": steps, "warmup": warm,
           "ms_per_step": modes["predict"]["ms_per_step"], "dtype": "i8",
           "config": {"workload": cfg.name, "format": fmt, "tokens": cfg.T, "layers": L, "hidden": cfg.C,
                      "experts": cfg.E, "top_k": cfg.k, "ffn": cfg.R, "resident_per_layer": cfg.resident,
                      "predictor": f"{cfg.C}->{cfg.pred_hidden}->{cfg.E}",
                      "experts_selected_per_layer": round(sum(active) / L, 2)},
           "staging": modes, "setup_s": round(build_s, 1),
           "kernels_us": {k: round(v[1] / v[0] * 1e3, 2) for k, v in prof.items() if v[0]},
           "roofline": stack_roofline(cfg, L, fmt, prof, active)}
    if cpu_s > 0:
        ld = stack.layers[0]
        res["cpu_baseline"] = cpu_baseline(cfg, dict(x=ld.x, wr=ld.w_router, bias=ld.bias), cpu_s, fmt)
    del stack
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def percentiles(us):
    """p10 / p50 / p90 of a list of per-call times in microseconds."""
    v = sorted(us)
    if not v:
        return None
    pick = lambda q: v[min(len(v) - 1, int(round(q * (len(v) - 1))))]
    return {"p10": round(pick(0.1), 2), "p50": round(pick(0.5), 2), "p90": round(pick(0.9), 2),
            "calls": len(v)}


def profiler_attached():
    """True under rocprofv3: its preloaded library initialises the GPU in
    every process it starts, so a child program must not be spawned then."""
    return any(k.startswith("ROCPROF") for k in os.environ) or "rocprofiler" in os.environ.get("LD_PRELOAD", "")


def smi_info():
    """Product name and clocks from rocm-smi.  Runs a child process, so it is
    called before this process touches the GPU, and skipped under a profiler."""
    import subprocess
    if profiler_attached():
        return {"product": "skipped (profiler attached)", "clocks": "skipped (profiler attached)"}
    info = {}
    for key, cmd in (("product", ["rocm-smi", "--showproductname", "--json"]),
                     ("clocks", ["rocm-smi", "--showclocks", "--json"])):
        try:
            r = subprocess.run(cmd, capture_output=True, text=True, timeout=20)
            card = next(iter(json.loads(r.stdout).values()))
            info[key] = {k.strip(" :"): v for k, v in card.items()}
        except Exception as e:  # informational only
            info[key] = f"unavailable ({type(e).__name__})"
    return info


def device_info(smi):
    """SKU, compute units, HBM and clocks of the GPU the bench runs on."""
    import torch
    pr = torch.cuda.get_device_properties(0)
    info = {"name": pr.name, "arch": getattr(pr, "gcnArchName", ""), "compute_units": pr.multi_processor_count,
            "hbm_gib": round(pr.total_memory / 2 ** 30, 1)}
    info.update(smi)
    return info


def copy_bandwidth(nbytes=1 << 30, reps=20):
    """Read + write GB/s of a plain device-to-device copy (the practical
    ceiling a streaming kernel is compared with), median of reps."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    times = []
    for i in range(reps + 3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        e1.synchronize()
        if i >= 3:
            times.append(e0.elapsed_time(e1) * 1e-3)
    times.sort()
    t = times[len(times) // 2]
    del src, dst
    torch.cuda.empty_cache()
    return round(2 * nbytes / t / 1e9, 1)


def run_layer(cfg, fmt, steps, warmup, cpu_s, prof_on=True, copy_gbs=None):
    """One workload's layer call: `steps` timed calls over rotating layer
    copies, the dominant kernel's roofline from its dispatch-recorded events,
    per-call p10/p50/p90 from a separate pass with an event pair around each
    call, and the oracle on a bounded sample (cpu_s seconds per leg; 0 =
    skip).  Returns the fields of the bench line."""
    import torch
    import paper_2609_38090_amd as mira

    # bytes of packed experts one call can touch: at most min(G, T*k + S) experts
    touched = min(cfg.G, cfg.T * cfg.k + cfg.S) * expert_stride(cfg, fmt)
    n_copies = max(2, min(8, math.ceil(COLD_BYTES / max(1, touched)) + 1))
    if cfg.name == "tiny":
        n_copies = 1
    copies, stride, act = build_copies(cfg, n_copies, fmt)
    shape = mira.MoEShape(cfg.C, cfg.R, cfg.E, cfg.k, cfg.S, act, format_flag(fmt))
    T = cfg.T
    ws = torch.empty(mira.mira_workspace_bytes(shape, T), dtype=torch.uint8, device="cuda")
    out = torch.empty((T, cfg.C), dtype=torch.float32, device="cuda")
    counts = torch.zeros((cfg.G,), dtype=torch.int32, device="cuda")
    argsets = []
    for c in copies:
        argsets.append(mira.MoEArgs(x=c["x"], n_tokens=T, n_slots=cfg.G, w_router=c["wr"],
                                    router_bias=c["bias"], slot_table=c["table"], slot_pool=c["pool"],
                                    slot_stride=stride, out=out, expert_counts=counts, workspace=ws,
                                    workspace_bytes=ws.numel()))
    stream = torch.cuda.current_stream()

    def step(i):
        mira.mira_moe_forward(shape, argsets[i % len(argsets)], stream)

    # routed counts of each copy (for the algorithmic byte / flop counts)
    units = []
    for i in range(len(argsets)):
        step(i)
        torch.cuda.synchronize()
        units.append(algorithmic_units(cfg, counts.cpu().tolist(), fmt))
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()

    decode = T <= mira.MIRA_DECODE_MAX_TOKENS
    dominant = "decode_gateup" if decode else "prefill_gateup"

    def sampled(i):
        return prof_on and event_step(i, len(argsets))

    if prof_on:
        # only the dominant kernel carries event records
        mira.mira_profile_select(dominant)
        mira.mira_profile_enable(False)
        mira.mira_profile_read()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        if sampled(i):
            mira.mira_profile_enable(True)
            step(i)
            mira.mira_profile_enable(False)
        else:
            step(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = mira.mira_profile_read() if prof_on else {}
    mira.mira_profile_select(None)

    # per-call distribution: a separate pass, one event pair around each call
    per_call = []
    n_dist = max(len(argsets) * 4, min(200, steps))
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_dist)]
    for i, (e0, e1) in enumerate(evs):
        e0.record(stream)
        step(i)
        e1.record(stream)
    torch.cuda.synchronize()
    per_call = [e0.elapsed_time(e1) * 1e3 for e0, e1 in evs]

    ms = elapsed * 1e3 / steps
    value = T / (ms / 1e3)
    # average algorithmic units per step over the rotation actually timed,
    # and over the steps whose dominant launch carried the events
    avg = {k: sum(units[i % len(units)][k] for i in range(steps)) / steps for k in units[0]}
    samp = [i for i in range(steps) if sampled(i)] or [0]
    avg_s = {k: sum(units[i % len(units)][k] for i in samp) / len(samp) for k in units[0]}
    roof = None
    cnt, tot = prof.get(dominant, (0, 0.0))
    if cnt:
        dur = tot / cnt * 1e-3
        if decode:
            achieved = avg_s["gu_bytes"] / dur / 1e9
            roof = {"bound": "hbm", "kernel": dominant, "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": traffic_bytes(dominant, cfg.name if fmt == "int8" else f"{cfg.name}_int4"),
                    "avg_us": round(dur * 1e6, 2),
                    "algorithmic_bytes_per_launch": int(avg_s["gu_bytes"]),
                    "timed_launches": cnt}
            if copy_gbs:
                roof["frac_of_copy"] = round(achieved / copy_gbs, 4)
        else:
            achieved = avg_s["gu_flops"] / dur / 1e12
            roof = {"bound": "mfma", "kernel": dominant, "achieved": round(achieved, 1),
                    "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(achieved / BF16_PEAK_TFLOPS, 4),
                    "traffic": traffic_bytes(dominant, cfg.name),
                    "avg_us": round(dur * 1e6, 2),
                    "algorithmic_flops_per_launch": avg_s["gu_flops"],
                    "achieved_hbm_gbs": round(avg_s["gu_bytes"] / dur / 1e9, 1),
                    "timed_launches": cnt}
    step_bytes = avg["gu_bytes"] + avg["dn_bytes"]
    res = {
        "value": round(value, 2),
        "unit": "tokens/s",
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms, 5),
        "dtype": "i8" if decode else "bf16",
        "config": {"workload": cfg.name, "format": fmt, "tokens": T, "hidden": cfg.C, "experts": cfg.E,
                   "top_k": cfg.k, "ffn": cfg.R, "shared_experts": cfg.S,
                   "activations": cfg.act, "layer_copies": len(copies),
                   "experts_touched_per_step": round(avg["active"], 2)},
        "per_call_us": dict(percentiles(per_call), note="separate pass, an event pair around each call"),
        "step_packed_gbs": round(step_bytes / (ms / 1e3) / 1e9, 1),
        "step_tflops": round((avg["gu_flops"] + avg["dn_flops"]) / (ms / 1e3) / 1e12, 2),
        "kernels_us": {k: round(v[1] / v[0] * 1e3, 2) for k, v in prof.items() if v[0]},
        "roofline": roof,
    }
    if cpu_s > 0:
        res["cpu_baseline"] = cpu_baseline(cfg, copies[0], cpu_s, fmt)
    del copies, argsets, ws, out
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        print("bench.py measures the MoE expert step on a single GPU; the library has no "
              "multi-GPU path (no sharding, no collectives).", file=sys.stderr)
        return 2

    if args.scale_bench:
        scale_bench()
        return 0

    if args.source_hash:
        print(json.dumps({f"{k[0]}/{k[1]}": source_hash(v["sources"]) for k, v in TRAFFIC.items()}))
        return 0
    if args.copy_bytes:
        return copy_reference(args.copy_bytes, args.steps)

    smi = smi_info()  # before anything touches the GPU
    import paper_2609_38090_amd as mira
    from mira_inputs import CONFIGS

    mira.load()
    name = args.workload or "mixtral_decode"
    cfg = CONFIGS[name]
    fmt = args.format
    if fmt == "int4" and cfg.T > mira.MIRA_DECODE_MAX_TOKENS:
        print(json.dumps({"error": "the INT4 variant runs on the decode kernels: use a decode "
                                   "workload (mixtral_decode, beam_stack, tiny)", "workload": cfg.name}))
        return 2
    if cfg.layers > 1:
        return run_stack(args, cfg)
    cpu_s = 0 if args.no_cpu_baseline else args.cpu_seconds
    copy_gbs = copy_bandwidth()
    res = run_layer(cfg, fmt, args.steps, args.warmup, cpu_s, not args.no_profile, copy_gbs)
    line = {"metric": METRIC, "value": res["value"], "unit": "tokens/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": res["ms_per_step"],
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": res["dtype"], "data": "synthetic"}
    line.update({k: v for k, v in res.items() if k not in line})
    line["device"] = device_info(smi)
    line["copy_gbs"] = copy_gbs
    line["paper_context"] = PAPER_CONTEXT
    if args.workload is None:
        # the default run also measures the prefill layers and the beam stack
        others = {}
        extra_cpu = 0 if args.no_cpu_baseline else args.extra_cpu_seconds
        for other in ("mixtral_prefill", "fine_grained"):
            print(f"[bench] {other}", file=sys.stderr, flush=True)
            others[other] = run_layer(CONFIGS[other], "int8", args.steps, args.warmup, extra_cpu,
                                      not args.no_profile)
        print("[bench] beam_stack", file=sys.stderr, flush=True)
        others["beam_stack"] = run_stack(args, CONFIGS["beam_stack"], summary=True, cpu_s=extra_cpu)
        line["workloads"] = others
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
