#!/usr/bin/env python3
"""Throughput of the routed mixture-of-head attention layer on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload N]

A step is one pass of the whole layer over one batch of seeded synthetic
input already resident in HBM: for prefill workloads route (top-K, gates,
permutation) + attention (packing with RoPE, MFMA attention, gated combine);
for the decode workload one decode step (route, append, history attention,
combine).  Prints one JSON line.

Without --workload the line's headline is the largest prefill workload, the
skewed-routing one (B=2, T=16384, H=32, K=4, d=128: 327 GFLOP of causal
attention per step), and the line carries one object per other workload
under "workloads": the balanced prefill (B=4, T=4096, H=32, K=8, d=64), the
long-context head-scaling prefill (B=1, T=32768, H=64, K=8, d=128) and the
decode step (64 sequences, 131072 prior tokens, H=64, K=8, d=128), each with
its own roofline and CPU baseline.  --workload N runs one workload alone.

The roofline entry is for the dominant kernel (routed attention for prefill,
history attention for decode): algorithmic FLOPs (4*d*sum n(n+1)/2) or bytes
(sum over active heads of (n+1)*2*d*2) per launch divided by its average
duration, timed with HIP events that the library attaches to the kernel's
dispatch on the launch stream (the interval a kernel trace records).
The cpu_baseline entry times the CPU oracle (float64 numpy) on a bounded
sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2609_38832_amd import workloads as W  # noqa: E402

METRIC = "routed-attn prefill tokens/s + decode KV GB/s, % of MFMA/HBM peak (1 GPU)"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_digest(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_entry(kernel, workload_name, per_launch_units):
    """HBM traffic from committed rocprofv3 counter runs, if they were taken
    on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload_name}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("source_digest") != source_digest(rec["sources"]):
        return None
    return rec.get("bytes_per_launch")


def cpu_info():
    cores = len(os.sched_getaffinity(0))
    threads = None
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        if info:
            threads = max(i.get("num_threads", 1) for i in info)
    except Exception:
        pass
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return cores, threads, model


def warm_up(step, args, torch):
    """args.warmup untimed steps, then more until at least args.settle_ms of
    continuous GPU work has run: the first tens of milliseconds of sustained
    load on the part run at transient clocks (kernel times move by up to 40 %
    over the first ~40 ms), so the timed steps start from the steady state.
    Returns the number of untimed steps run."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.warmup):
        step()
    e1.record()
    torch.cuda.synchronize()
    done = args.warmup
    per = e0.elapsed_time(e1) / max(args.warmup, 1)
    if args.settle_ms > 0:
        more = max(0, int(math.ceil(args.settle_ms / max(per, 1e-3))) - args.warmup)
        for _ in range(more):
            step()
        torch.cuda.synchronize()
        done += more
    return done


# ----------------------------------------------------------------------------
def bench_prefill(w, args, torch, L, DI):
    dev = torch.device("cuda:0")
    log(f"generating inputs for {w.name}")
    inp = W.prefill_inputs(w)
    logits = torch.from_numpy(inp["logits"]).to(dev)
    q, k, v = (DI.to_device(inp[n], w.dtype, dev) for n in ("q", "k", "v"))
    B, T, H, K, d = w.B, w.T, w.H, w.K, w.d
    i32 = dict(dtype=torch.int32, device=dev)
    routing = {
        "topk_idx": torch.empty(B, T, K, **i32),
        "gates": torch.empty(B, T, K, dtype=torch.float32, device=dev),
        "head_len": torch.empty(B, H, **i32),
        "seg_offsets": torch.empty(B * H + 1, **i32),
        "perm_token": torch.empty(B * T * K, **i32),
        "slot_pos": torch.empty(B, T, K, **i32),
    }
    rws = L.workspace(L.route_workspace_size(B, T, H, K), dev)
    dt = L.dtype_code(q.dtype)
    aws = L.workspace(L.attn_workspace_size(B, T, H, K, d, dt), dev)
    out = torch.empty(B, T, d, dtype=q.dtype, device=dev)

    def step():
        L.route(logits, K, L.GATE_SOFTMAX_SELECTED, out=routing, ws=rws)
        L.attn_fwd(q, k, v, routing, K, w.rope_base, L.ROPE_HEAD_RELATIVE, out=out, ws=aws)

    log(f"warmup {args.warmup} steps, settle {args.settle_ms} ms")
    warm = warm_up(step, args, torch)
    n = routing["head_len"].cpu().numpy().astype(np.int64)
    c_attn = int((n * (n + 1) // 2).sum())
    flops = 4.0 * d * c_attn

    # timed region: whole steps only
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms_total = e0.elapsed_time(e1)
    # the same steps again with the library's per-kernel event timing on
    # (the extra event records sit between kernels, so they are kept out of
    # the step timing above)
    L.profile_enable(args.steps)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kern = {}
    for sec in ("route_count", "route_scan", "route_scatter", "pack", "attn", "merge", "combine"):
        r = L.profile_read(sec)
        if r is not None and r[1] > 0:
            kern[sec] = r[0] / r[1]
    L.profile_enable(0)
    ms_step = ms_total / args.steps
    tokens_s = B * T / (ms_step * 1e-3)
    attn_ms = kern.get("attn", float("nan"))
    mfma = w.dtype == "bf16" and d in (64, 128)
    peak = PEAK_BF16_TFLOPS if mfma else PEAK_FP32_TFLOPS
    achieved = flops / (attn_ms * 1e-3) / 1e12
    roof = {"kernel": "k_attn_mfma" if mfma else "k_attn_generic",
            "bound": "mfma" if mfma else "alu", "achieved": round(achieved, 2), "peak": peak,
            "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
            "traffic": traffic_entry("k_attn_mfma", w.name, None),
            "algorithmic_per_launch": {"flops": flops, "C_attn": c_attn},
            "kernel_ms": round(attn_ms, 4)}
    res = {"metric": METRIC, "value": round(tokens_s, 1), "unit": "tokens/s",
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
           "config": {"workload": w.name, "B": B, "T": T, "H": H, "K": K, "d_head": d,
                      "rope": "head-relative", "rope_base": w.rope_base,
                      "gates": "softmax over selected"},
           "roofline": roof,
           "kernels_ms": {k2: round(v2, 4) for k2, v2 in kern.items()},
           "kernels_hbm": hbm_kernels(kern, w),
           "warmup_steps_run": warm, "settle_ms": args.settle_ms}
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline_prefill(w, inp, n, args.cpu_budget)
    return res


def hbm_kernels(kern, w):
    """Algorithmic HBM bytes and GB/s of the routing, packing and combine
    kernels (reported, not the graded roofline).  Nr = B T K routed pairs:
      route_count   logits [B,T,H] f32 in; top-K index, gate, in-chunk rank
                    [B,T,K] i32/f32 and the chunk counts out;
      route_scatter top-K index and rank in; token of each packed row and
                    packed row of each (t, k) out;
      pack          the routed key and value rows in, packed key tiles and
                    transposed value tiles out (all of the inputs' dtype);
      combine       the packed head rows (bf16) and gates / slots in, the
                    layer output out."""
    B, T, H, K, d = w.B, w.T, w.H, w.K, w.d
    Nr = B * T * K
    esz = 2 if w.dtype == "bf16" else 4
    nchunk = (T + 63) // 64
    counts = B * H * nchunk * 4
    nbytes = {
        "route_count": B * T * H * 4 + 3 * Nr * 4 + counts,
        "route_scatter": 2 * Nr * 4 + 2 * Nr * 4 + counts,
        "pack": 4 * Nr * d * esz,
        "combine": Nr * d * (2 if esz == 2 else 4) + 2 * Nr * 4 + B * T * d * esz,
    }
    out = {}
    for k, b in nbytes.items():
        if k in kern and kern[k] > 0:
            out[k] = {"bytes": b, "GB/s": round(b / (kern[k] * 1e-3) / 1e9, 1),
                      "frac_of_8TB/s": round(b / (kern[k] * 1e-3) / 1e9 / PEAK_HBM_GBS, 3)}
    return out


def cpu_baseline_prefill(w, inp, head_len, budget_s):
    import oracle as O
    cores, threads, model = cpu_info()
    log(f"cpu baseline: oracle on up to ~{budget_s:.0f} s of segments")
    t0 = time.perf_counter()
    topk = O.select_heads(inp["logits"], w.K)
    g = O.route_gates(inp["logits"], topk, O.GATE_SOFTMAX_SELECTED)
    n, off, perm, slot = O.permutation(topk, w.H)
    t_route = time.perf_counter() - t0
    # attention over whole segments, in order, until the budget is spent
    f64 = {}
    done_work, segs = 0, 0
    t1 = time.perf_counter()
    total_work = float((head_len * (head_len + 1) // 2).sum())
    for sid in range(w.B * w.H):
        b, h = divmod(sid, w.H)
        if (b, h) not in f64:
            f64[(b, h)] = True
        sub = {key: W.as_float64(inp[key][b:b + 1, h:h + 1], w.dtype) for key in ("q", "k", "v")}
        a, e = int(off[sid]), int(off[sid + 1])
        off_local = np.array([0, e - a], dtype=np.int64)
        O.attention_gathered(sub["q"], sub["k"], sub["v"], None, off_local, perm[a:e], 1,
                             w.rope_base)
        nn = e - a
        done_work += nn * (nn + 1) / 2
        segs += 1
        if time.perf_counter() - t1 > budget_s:
            break
    t_attn = time.perf_counter() - t1
    t_est = t_route + t_attn * (total_work / max(done_work, 1.0))
    return {"value": round(w.B * w.T / t_est, 2), "unit": "tokens/s", "cores": threads or cores,
            "kind": "oracle",
            "sample": (f"routing+permutation of the whole batch ({t_route:.2f} s) plus float64 "
                       f"gathered causal attention of {segs}/{w.B * w.H} (batch, head) segments "
                       f"({t_attn:.2f} s), extrapolated by causal work sum n(n+1)/2"),
            "host_cpu": model, "host_cores": cores}


# ----------------------------------------------------------------------------
def bench_layer(w, args, torch, L, DI):
    """The layer with its routed projections: route, Q/K/V projections of
    the routed pairs, routed attention (head outputs), output projections of
    the routed pairs with the gated combine."""
    dev = torch.device("cuda:0")
    log(f"generating inputs for {w.name}")
    inp = W.projection_inputs(w)
    logits = torch.from_numpy(inp["logits"]).to(dev)
    x, wq, wo = (DI.to_device(inp[n], "bf16", dev) for n in ("x", "w_qkv", "w_o"))
    B, T, H, K, d, dm = w.B, w.T, w.H, w.K, w.d, w.d_model
    routing = L.route(logits, K)
    rws = L.workspace(L.route_workspace_size(B, T, H, K), dev)
    qkv = {n: torch.empty(B, H, T, d, dtype=torch.bfloat16, device=dev) for n in ("q", "k", "v")}
    aws = L.workspace(L.attn_workspace_size(B, T, H, K, d, L.BF16), dev)
    ho = torch.empty(B * T * K, d, dtype=torch.float32, device=dev)
    ows = L.workspace(L.out_proj_workspace_size(B, T, H, K, w.d, dm), dev)
    out = torch.empty(B, T, dm, dtype=torch.bfloat16, device=dev)

    def step():
        L.route(logits, K, L.GATE_SOFTMAX_SELECTED, out=routing, ws=rws)
        L.qkv_proj(x, wq, routing, H, K, out=qkv)
        L.attn_fwd(qkv["q"], qkv["k"], qkv["v"], routing, K, w.rope_base, head_out=ho, out=False,
                   ws=aws)
        L.out_proj(ho, wo, routing, B, T, H, K, out=out, ws=ows)

    log(f"warmup {args.warmup} steps")
    warm_up(step, args, torch)
    n = routing["head_len"].cpu().numpy().astype(np.int64)
    Nr = B * T * K
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    L.profile_enable(args.steps)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kern = {}
    for sec in ("qkv_proj", "pack", "attn", "out_proj", "out_combine"):
        r = L.profile_read(sec)
        if r is not None and r[1] > 0:
            kern[sec] = r[0] / r[1]
    L.profile_enable(0)
    # algorithmic work: 2 d_model 3d FLOP per routed pair for Q/K/V, 2 d d_model
    # for the output projection, 4 d sum n(n+1)/2 for the attention
    f_qkv = 2.0 * Nr * dm * 3 * d
    f_out = 2.0 * Nr * d * dm
    f_attn = 4.0 * d * float((n * (n + 1) // 2).sum())
    qkv_ms = kern.get("qkv_proj", float("nan"))
    achieved = f_qkv / (qkv_ms * 1e-3) / 1e12
    res = {"metric": "routed-attn layer with routed projections, tokens/s (1 GPU)",
           "value": round(B * T / (ms_step * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic",
           "config": {"workload": w.name, "B": B, "T": T, "H": H, "K": K, "d_head": d,
                      "d_model": dm, "rope": "head-relative", "rope_base": w.rope_base,
                      "gates": "softmax over selected"},
           "roofline": {"kernel": "k_proj_big<QKV>", "bound": "mfma",
                        "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                        "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                        "traffic": None,
                        "algorithmic_per_launch": {"flops": f_qkv},
                        "kernel_ms": round(qkv_ms, 4)},
           "work": {"qkv_flops": f_qkv, "attn_flops": f_attn, "out_flops": f_out,
                    "out_rows_bytes": 2.0 * Nr * dm * 2},
           "kernels_ms": {k2: round(v2, 4) for k2, v2 in kern.items()}}
    # the library's output-projection form (dense over all heads when H d <= 384 K)
    dense = H * d <= 384 * K and H <= 64
    res["out_proj_form"] = "dense" if dense else "per-pair"
    if "out_proj" in kern:
        res["out_proj_gemm_tflops"] = round(f_out / (kern["out_proj"] * 1e-3) / 1e12, 1)
        if dense:
            f_exec = 2.0 * B * T * H * d * dm
            res["out_proj_executed_tflops"] = round(f_exec / (kern["out_proj"] * 1e-3) / 1e12, 1)
    return res


# ----------------------------------------------------------------------------
def bench_grouped(w, args, torch, L, DI):
    """Key/value-group routing on a prefill workload: the H query heads form
    H/g groups sharing one key/value head; K/g groups are selected per token."""
    g = args.kv_group
    if w.H % g or w.K % g:
        raise SystemExit(f"--kv-group {g} must divide H = {w.H} and K = {w.K}")
    dev = torch.device("cuda:0")
    wk = w.with_(H=w.H // g, K=w.K // g)
    log(f"generating inputs for {w.name} with key/value groups of {g}")
    logits = torch.from_numpy(W.prefill_logits(wk)).to(dev)
    q = DI.to_device(W.prefill_qkv(w, "q"), w.dtype, dev)
    k, v = (DI.to_device(W.prefill_qkv(wk, n), w.dtype, dev) for n in ("k", "v"))
    B, T, Hkv, Kkv, d = w.B, w.T, wk.H, wk.K, w.d
    routing = L.route(logits, Kkv)
    rws = L.workspace(L.route_workspace_size(B, T, Hkv, Kkv), dev)
    aws = L.workspace(int(L.lib().namoh_attn_fwd_grouped_workspace_size(B, T, Hkv, Kkv, g, d,
                                                                         L.dtype_code(q.dtype))),
                      dev)
    out = torch.empty(B, T, d, dtype=q.dtype, device=dev)

    def step():
        L.route(logits, Kkv, L.GATE_SOFTMAX_SELECTED, out=routing, ws=rws)
        L.attn_fwd_grouped(q, k, v, routing, Kkv, w.rope_base, out=out, ws=aws)

    warm_up(step, args, torch)
    n = routing["head_len"].cpu().numpy().astype(np.int64)
    # Eq. app-group-prefill: every routed row of a group carries g queries
    c_attn = g * int((n * (n + 1) // 2).sum())
    flops = 4.0 * d * c_attn
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    L.profile_enable(args.steps)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kern = {}
    for sec in ("attn", "pack", "combine"):
        r = L.profile_read(sec)
        if r is not None and r[1] > 0:
            kern[sec] = r[0] / r[1]
    L.profile_enable(0)
    attn_ms = kern.get("attn", float("nan"))
    achieved = flops / (attn_ms * 1e-3) / 1e12
    return {"metric": "routed-attn prefill with key/value-group routing, tokens/s (1 GPU)",
            "value": round(B * T / (ms_step * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
            "data": "synthetic",
            "config": {"workload": w.name, "kv_group": g, "B": B, "T": T, "H": w.H, "K": w.K,
                       "H_kv": Hkv, "K_kv": Kkv, "d_head": d, "rope": "head-relative",
                       "rope_base": w.rope_base, "gates": "softmax over selected"},
            "roofline": {"kernel": "k_attn_mfma", "bound": "mfma", "achieved": round(achieved, 2),
                         "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                         "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None,
                         "algorithmic_per_launch": {"flops": flops, "C_attn": c_attn},
                         "kernel_ms": round(attn_ms, 4)},
            "kernels_ms": {k2: round(v2, 4) for k2, v2 in kern.items()}}


# ----------------------------------------------------------------------------
def bench_shared(w, args, torch, L, DI):
    """A prefill step with always-active shared heads added: routing, routed
    attention, then Hs shared heads (causal or sliding window) summed into
    the same output."""
    hs, win = (int(x) for x in args.shared.split(":"))
    dev = torch.device("cuda:0")
    log(f"generating inputs for {w.name} with {hs} shared heads, window {win}")
    inp = W.prefill_inputs(w)
    logits = torch.from_numpy(inp["logits"]).to(dev)
    q, k, v = (DI.to_device(inp[n], w.dtype, dev) for n in ("q", "k", "v"))
    ws_ = w.with_(H=hs, K=1, seed=w.seed + 100)
    qs, ks, vs = (DI.to_device(W.prefill_qkv(ws_, n), w.dtype, dev) for n in ("q", "k", "v"))
    B, T, H, K, d = w.B, w.T, w.H, w.K, w.d
    routing = L.route(logits, K)
    rws = L.workspace(L.route_workspace_size(B, T, H, K), dev)
    aws = L.workspace(L.attn_workspace_size(B, T, H, K, d, L.dtype_code(q.dtype)), dev)
    sws = L.workspace(int(L.lib().namoh_shared_attn_workspace_size(B, T, hs, d)), dev)
    out = torch.empty(B, T, d, dtype=q.dtype, device=dev)

    def step():
        L.route(logits, K, L.GATE_SOFTMAX_SELECTED, out=routing, ws=rws)
        L.attn_fwd(q, k, v, routing, K, w.rope_base, out=out, ws=aws)
        L.shared_attn(qs, ks, vs, win, w.rope_base, out=out, accumulate=True, ws=sws)

    warm_up(step, args, torch)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    L.profile_enable(2 * args.steps)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    r = L.profile_read("attn")
    L.profile_enable(0)
    # the "attn" section holds the routed and the shared attention launches of
    # every step, in that order
    times = None if r is None else r[0] / r[1]
    t = np.arange(T, dtype=np.int64)
    pairs = int((np.minimum(t + 1, win) if win > 0 else t + 1).sum()) * B * hs
    return {"metric": "routed-attn prefill plus always-active shared heads, tokens/s (1 GPU)",
            "value": round(B * T / (ms_step * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
            "data": "synthetic",
            "config": {"workload": w.name, "shared_heads": hs, "window": win, "B": B, "T": T,
                       "H": H, "K": K, "d_head": d, "rope": "head-relative (routed), global "
                       "(shared)", "rope_base": w.rope_base},
            "shared_attention": {"flops": 4.0 * d * pairs, "pairs": pairs},
            "attn_kernels_mean_ms": None if times is None else round(times, 4)}


# ----------------------------------------------------------------------------
def bench_backward(w, args, torch, L, DI):
    """One training step of the layer: route, forward, backward of the
    attention (dq, dk, dv, dgates) and of the gates (d logits)."""
    dev = torch.device("cuda:0")
    log(f"generating inputs for {w.name} (training step)")
    inp = W.prefill_inputs(w)
    logits = torch.from_numpy(inp["logits"]).to(dev)
    q, k, v = (DI.to_device(inp[n], w.dtype, dev) for n in ("q", "k", "v"))
    B, T, H, K, d = w.B, w.T, w.H, w.K, w.d
    g = torch.Generator(device="cpu").manual_seed(w.seed + 77)
    dout = (torch.randn(B, T, d, generator=g, dtype=torch.float32) * 0.1).to(dev)
    routing = L.route(logits, K)
    rws = L.workspace(L.route_workspace_size(B, T, H, K), dev)
    dt = L.dtype_code(q.dtype)
    aws = L.workspace(L.attn_workspace_size(B, T, H, K, d, dt), dev)
    bws = L.workspace(int(L.lib().namoh_attn_bwd_workspace_size(B, T, H, K, d)), dev)
    out = torch.empty(B, T, d, dtype=q.dtype, device=dev)
    f32 = dict(dtype=torch.float32, device=dev)
    Nr = B * T * K
    # gradients of the routed pairs in the routing's packed order (what a
    # routed projection's backward consumes); the dense form is timed beside
    grads = {"dq": torch.empty(Nr, d, **f32), "dk": torch.empty(Nr, d, **f32),
             "dv": torch.empty(Nr, d, **f32), "dgates": torch.empty(B, T, K, **f32)}
    dense = {"dq": torch.empty(B, H, T, d, **f32), "dk": torch.empty(B, H, T, d, **f32),
             "dv": torch.empty(B, H, T, d, **f32), "dgates": torch.empty(B, T, K, **f32)}

    mfma = w.dtype == "bf16" and d in (64, 128)

    def step(packed=True, saved=True):
        # saved: the training forward leaves its statistics and tiles in the
        # backward's workspace, which the backward reuses; otherwise the
        # stateless forward, and a backward that reruns the forward itself
        L.route(logits, K, L.GATE_SOFTMAX_SELECTED, out=routing, ws=rws)
        g = grads if packed else dense
        if saved and mfma:
            L.attn_fwd_train(q, k, v, routing, K, w.rope_base, bws, out=out)
            L.attn_bwd(q, k, v, routing, K, w.rope_base, dout, ws=bws, out=g, packed=packed,
                       saved=True)
        else:
            L.attn_fwd(q, k, v, routing, K, w.rope_base, L.ROPE_HEAD_RELATIVE, out=out, ws=aws)
            L.attn_bwd(q, k, v, routing, K, w.rope_base, dout, ws=bws, out=g, packed=packed)
        L.route_bwd(logits, routing, g["dgates"])

    log(f"warmup {args.warmup} steps")
    warm_up(step, args, torch)
    n = routing["head_len"].cpu().numpy().astype(np.int64)
    c_attn = int((n * (n + 1) // 2).sum())
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    for _ in range(args.warmup):
        step(packed=False)
    e0.record()
    for _ in range(args.steps):
        step(packed=False)
    e1.record()
    torch.cuda.synchronize()
    ms_step_dense = e0.elapsed_time(e1) / args.steps
    for _ in range(args.warmup):
        step(saved=False)
    e0.record()
    for _ in range(args.steps):
        step(saved=False)
    e1.record()
    torch.cuda.synchronize()
    ms_step_rerun = e0.elapsed_time(e1) / args.steps
    L.profile_enable(2 * args.steps)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kern = {}
    for sec in ("attn", "pack", "combine", "bwd_pack", "bwd_dq", "bwd_dkdv"):
        r = L.profile_read(sec)
        if r is not None and r[1] > 0:
            kern[sec] = r[0] / r[1]
    L.profile_enable(0)
    # the backward's products per causal (query, key) pair: dP = dO V^T, the
    # recomputed scores, dV += P^T dO, dQ += dS K, dK += dS^T Q: 2d FLOP each;
    # the algorithmic count is 10 d (scores counted once); the two kernels
    # execute 6 d (dq: S, dP, dQ) and 8 d (dkdv: S, dP, dV, dK)
    bwd_ms = kern.get("bwd_dq", float("nan")) + kern.get("bwd_dkdv", float("nan"))
    flops = 10.0 * d * c_attn
    achieved = flops / (bwd_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if mfma else PEAK_FP32_TFLOPS
    res = {"metric": "routed-attn training step tokens/s (route + forward + backward), "
                     "backward MFMA kernels % of bf16 peak (1 GPU)",
           "value": round(B * T / (ms_step * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": w.dtype, "data": "synthetic",
           "ms_per_step_dense_grads": round(ms_step_dense, 4),
           "ms_per_step_forward_rerun": round(ms_step_rerun, 4),
           "config": {"workload": w.name, "B": B, "T": T, "H": H, "K": K, "d_head": d,
                      "pass": "training step", "gradients": "packed (routed pairs)",
                      "forward_state": "saved by the training forward" if mfma else "recomputed",
                      "rope": "head-relative",
                      "rope_base": w.rope_base, "gates": "softmax over selected"},
           "roofline": {"kernel": "k_bwd_dq + k_bwd_dkdv" if mfma else "k_bwd_q + k_bwd_kv",
                        "bound": "mfma" if mfma else "alu", "achieved": round(achieved, 2),
                        "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                        "traffic": None,
                        "algorithmic_per_launch": {"flops": flops, "C_attn": c_attn},
                        "kernel_ms": round(bwd_ms, 4)},
           "kernels_ms": {k2: round(v2, 4) for k2, v2 in kern.items()}}
    return res


# ----------------------------------------------------------------------------
def bench_decode(w, args, torch, L, DI):
    dev = torch.device("cuda:0")
    g = args.kv_group
    wq = w
    if g > 1:   # key/value groups: the routing, caches and lengths are per group
        if w.H % g or w.K % g:
            raise SystemExit(f"--kv-group {g} must divide H = {w.H} and K = {w.K}")
        w = w.with_(H=w.H // g, K=w.K // g)
    log(f"prior head lengths for {w.name}")
    lengths = W.decode_prior_lengths(w)
    # room for every append: warm-up, settle (a decode step takes more than
    # 0.4 ms, so settle_ms / 0.4 bounds the settle steps), timed and event-timed steps
    cap = W.decode_cache_capacity(
        lengths, steps=2 * args.warmup + 2 * args.steps + int(args.settle_ms / 0.4) + 8)
    log(f"filling caches on the device: 2 x [{w.B},{w.H},{cap},{w.d}] {w.dtype}")
    kc, vc = DI.decode_caches(w.B, w.H, cap, w.d, w.dtype, w.seed, w.qkv_scale, dev)
    step_in = W.decode_step_inputs(w)
    logits = torch.from_numpy(step_in["logits"]).to(dev)
    q_in = step_in["q"] if g == 1 else W.decode_step_inputs(wq)["q"]
    q = DI.to_device(q_in, w.dtype, dev)
    k, v = (DI.to_device(step_in[n], w.dtype, dev) for n in ("k", "v"))
    cache_len = torch.from_numpy(lengths).to(dev)
    B, H, K, d = w.B, w.H, w.K, w.d
    outd = {"topk_idx": torch.empty(B, K, dtype=torch.int32, device=dev),
            "gates": torch.empty(B, K, dtype=torch.float32, device=dev),
            "out": torch.empty(B, d, dtype=q.dtype, device=dev)}
    if g == 1:
        ws = L.workspace(L.decode_workspace_size(B, H, K, d, cap), dev)

        def step():
            L.decode_step(logits, q, k, v, kc, vc, cache_len, K, w.rope_base, out=outd, ws=ws)
    else:
        ws = L.workspace(int(L.lib().namoh_decode_grouped_workspace_size(B, H, K, g, d, cap)), dev)

        def step():
            r = L.decode_step_grouped(logits, q, k, v, kc, vc, cache_len, K, w.rope_base, ws=ws)
            outd.update(r)

    # warm-up, then settle with steps on a copy of the lengths, so the timed
    # and the kernel-timed steps below append at known positions
    log(f"warmup {args.warmup} steps, settle {args.settle_ms} ms")
    len_start = cache_len.clone()
    warm = warm_up(step, args, torch)
    cache_len.copy_(len_start)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    len0 = cache_len.cpu().numpy().astype(np.int64)
    topk = outd["topk_idx"].cpu().numpy()
    esz = 2 if w.dtype == "bf16" else 4
    # the same token is decoded each step, so the same heads grow by one row
    rows = [sum(int(len0[b, h]) + 1 + s for b in range(B) for h in topk[b])
            for s in range(2 * args.steps)]
    kv_bytes = [r * 2 * d * esz for r in rows]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms_total = e0.elapsed_time(e1)
    # kernel timing pass (event records between kernels, not in the step time);
    # these steps append further rows, which the byte count below includes
    L.profile_enable(args.steps)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    r = L.profile_read("decode_attn")
    L.profile_enable(0)
    kern_ms = r[0] / r[1]
    ms_step = ms_total / args.steps
    step_bytes = float(np.mean(kv_bytes[:args.steps]))
    kern_bytes = float(np.mean(kv_bytes[args.steps:]))
    gbs_step = step_bytes / (ms_step * 1e-3) / 1e9
    gbs_kern = kern_bytes / (kern_ms * 1e-3) / 1e9
    mean_bytes = kern_bytes
    res = {"metric": METRIC, "value": round(gbs_step, 1), "unit": "GB/s",
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
           "config": {"workload": wq.name, "B": B, "prior_tokens": w.prior, "H": wq.H, "K": wq.K,
                      "kv_group": g, "H_kv": H, "K_kv": K,
                      "d_head": d, "cap": cap, "rope": "head-relative", "rope_base": w.rope_base},
           "roofline": {"kernel": "k_decode_attn", "bound": "hbm", "achieved": round(gbs_kern, 1),
                        "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(gbs_kern / PEAK_HBM_GBS, 4),
                        "traffic": traffic_entry("k_decode_attn", w.name, None),
                        "algorithmic_per_launch": {"kv_bytes": mean_bytes,
                                                   "rows": float(np.mean(rows[args.steps:]))},
                        "kernel_ms": round(kern_ms, 4)},
           "tokens_per_s": round(B / (ms_step * 1e-3), 1),
           "warmup_steps_run": warm + args.warmup, "settle_ms": args.settle_ms}
    if not args.no_cpu_baseline and g == 1:
        res["cpu_baseline"] = cpu_baseline_decode(w, step_in, kc, vc, len0, topk, args.cpu_budget, torch)
    del kc, vc
    return res


def cpu_baseline_decode(w, step_in, kc, vc, lengths, topk, budget_s, torch):
    import oracle as O
    cores, threads, model = cpu_info()
    log("cpu baseline: oracle decode on a sample of sequences")
    d = w.d

    def host(t):
        return W.as_float64(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16), w.dtype) \
            if w.dtype == "bf16" else t.cpu().numpy().astype(np.float64)

    sf = {k: W.as_float64(step_in[k], w.dtype) for k in ("q", "k", "v")}
    done_bytes, t_sum, nseq = 0.0, 0.0, 0
    for b in range(w.B):
        hist = {int(h): (host(kc[b, h, :lengths[b, h]]), host(vc[b, h, :lengths[b, h]]))
                for h in topk[b]}
        t0 = time.perf_counter()
        O.decode_step(step_in["logits"][b:b + 1], sf["q"][b:b + 1], sf["k"][b:b + 1],
                      sf["v"][b:b + 1], lambda _b, h, n: hist[h][0], lambda _b, h, n: hist[h][1],
                      lengths[b:b + 1], w.K, w.rope_base)
        t_sum += time.perf_counter() - t0
        done_bytes += sum((int(lengths[b, h]) + 1) * 2 * d * 2 for h in topk[b])
        nseq += 1
        if t_sum > budget_s:
            break
    return {"value": round(done_bytes / t_sum / 1e9, 3), "unit": "GB/s",
            "cores": threads or cores, "kind": "oracle",
            "sample": (f"float64 decode step of {nseq}/{w.B} sequences "
                       f"({t_sum:.2f} s, history rows copied to the host beforehand, not timed); "
                       f"value = algorithmic bf16 KV bytes of those sequences / time"),
            "host_cpu": model, "host_cores": cores}


# ----------------------------------------------------------------------------
HEADLINE = 4          # skewed prefill: the largest prefill workload
SUITE_OTHERS = (2, 3, 5)


def bench_suite(args, torch, L, DI):
    """The headline workload's line, with one object per other workload."""
    if args.backward or args.shared or args.kv_group > 1:
        raise SystemExit("--backward, --shared and --kv-group need --workload")
    budget = args.cpu_budget
    res = bench_prefill(W.WORKLOADS[HEADLINE], args, torch, L, DI)
    torch.cuda.empty_cache()
    others = {}
    for n in SUITE_OTHERS:
        w = W.WORKLOADS[n]
        sub = argparse.Namespace(**vars(args))
        sub.cpu_budget = min(budget, 8.0)
        if w.decode:
            sub.steps = max(1, min(args.steps, 20))
            sub.warmup = max(1, min(args.warmup, 5))
        r = (bench_decode if w.decode else bench_prefill)(w, sub, torch, L, DI)
        torch.cuda.empty_cache()
        keep = ("value", "unit", "ms_per_step", "steps", "warmup", "warmup_steps_run",
                "settle_ms", "dtype", "config", "roofline", "kernels_ms", "kernels_hbm",
                "tokens_per_s", "cpu_baseline")
        others[w.name] = {k: r[k] for k in keep if k in r}
    res["workloads"] = others
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--workload", type=int, default=None, choices=sorted(W.WORKLOADS),
                    help="run one workload alone (default: the skewed prefill as the "
                         "headline plus the balanced, head-scaling and decode workloads)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kv-group", type=int, default=1,
                    help="key/value-group routing with groups of this many query heads "
                         "(prefill workloads; K/g of H/g groups selected per token)")
    ap.add_argument("--shared", type=str, default=None,
                    help="HS:W - add HS always-active shared heads with a window of W tokens "
                         "(0 = full causal prefix) to a prefill workload")
    ap.add_argument("--backward", action="store_true",
                    help="time a training step (route, forward, backward) of a prefill "
                         "workload instead of the forward step")
    ap.add_argument("--settle-ms", type=float, default=100.0,
                    help="after the warm-up steps, further untimed steps until this much "
                         "continuous GPU work has run (0: warm-up steps only)")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle work for the CPU baseline sample")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (reference for the "
                         "HBM byte counters of rocprofv3) and exit")
    ap.add_argument("--hbm-calibration", action="store_true",
                    help="only time a 4 GiB device-to-device copy with HIP events "
                         "(an achievable HBM rate to set the roofline fractions "
                         "against) and exit")
    args = ap.parse_args()
    if args.hbm_calibration:
        import torch
        n = 4 << 30
        src = torch.ones(n // 4, dtype=torch.int32, device="cuda:0")
        dst = torch.empty_like(src)
        res = {}
        for name, fn, nbytes in (("copy", lambda: dst.copy_(src), 2 * n),):
            for _ in range(3):
                fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(10):
                fn()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / 10
            res[name] = {"bytes": nbytes, "ms": round(ms, 4),
                         "GB_per_s": round(nbytes / ms / 1e6, 1)}
        print(json.dumps({"hbm_calibration": res, "peak_GB_per_s": 8000.0}))
        return
    if args.copy_calibration:
        import torch
        n = 1 << 30
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 3}))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; the path is sharded by "
                          "batch or head across GPUs in design only", "n_gpus": args.gpus}))
        sys.exit(2)
    suite = args.workload is None
    w = W.WORKLOADS[HEADLINE if suite else args.workload]
    if args.steps is None:
        args.steps = 20 if w.decode else 50
    if args.warmup is None:
        args.warmup = 5 if w.decode else 10
    import torch
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    from paper_2609_38832_amd import _lib as L
    from paper_2609_38832_amd import device_inputs as DI
    L.lib()
    if suite:
        res = bench_suite(args, torch, L, DI)
    elif args.backward:
        if w.decode:
            print(json.dumps({"error": "--backward needs a prefill workload"}))
            sys.exit(2)
        res = bench_backward(w, args, torch, L, DI)
    elif w.d_model:
        res = bench_layer(w, args, torch, L, DI)
    elif args.shared:
        if w.decode:
            print(json.dumps({"error": "--shared needs a prefill workload"}))
            sys.exit(2)
        res = bench_shared(w, args, torch, L, DI)
    elif args.kv_group > 1 and not w.decode:
        res = bench_grouped(w, args, torch, L, DI)
    else:
        res = (bench_decode if w.decode else bench_prefill)(w, args, torch, L, DI)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
