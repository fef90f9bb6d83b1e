#!/usr/bin/env python3
"""Decode-step benchmark of the KV-Direct hot path on one MI355X.

A step is one decode token of a Gemma-3-4B-shaped model (d=2560, 8 query / 4 KV
heads, head_dim 256, 34 layers, bf16), batch 1, 4096 checkpointed context
tokens per layer, with synthetic seeded residuals and random-init weights.
Per layer the step runs the whole hot path through libkvd's C ABI:

  kvd_project_qkv           q and the current token's K_t/V_t (RMSNorm, W_q/W_k/W_v, RoPE)
  kvd_fused_recompute_attn  K/V of the 4096 context tokens recomputed from the residual
                            checkpoints (RMSNorm, W_k/W_v GEMM, RoPE) into LDS, split-K
                            attention over [context || current token]; the workgroup that
                            completes a (sequence, KV head) merges its partials in-kernel

Printed: ONE JSON line with
  - tokens/s of the step, ms per step, and the roofline of the fused kernel from
    HIP events over the timed region;
  - per-op us/layer, and the cached-K/V and unfused baselines of the same step;
  - the recompute-vs-cached-read crossover over batch size (Gemma-3-4B layer,
    context 2048, B = 1..64; each op timed after a cache-evicting read), against a
    K/V cache in HBM and against one held in pinned host memory (copied over PCIe);
  - workloads: the SmolLM2-135M fp32 layer, the Qwen2.5-1.5B-shaped 28-layer step
    (B = 8, context 16384) and the Gemma-3-4B multi-turn step (B = 16, turn
    boundaries up to 5120 tokens), fused against cached;
  - cpu_baseline: the fp64 oracle on the host cores for the headline step, and
    cpu_baselines: bounded oracle samples of one layer of each other workload.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MI355X_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 MFMA
MI355X_HBM_PEAK_GBS = 8000.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "fused_kernel_traffic.json")
KERNEL_SOURCES = ["kvd_device.hpp", "kvd_kernels.hip", "kvd_layout.h"]


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-crossover", action="store_true")
    p.add_argument("--no-baselines", action="store_true", help="skip the cached / unfused per-op timings")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="CPU oracle time budget")
    p.add_argument("--sweep-batches", default="1,2,4,8,16,32,64")
    p.add_argument("--no-host-cache", action="store_true",
                   help="crossover without its host-resident cache leg (profiles count the attention dispatches "
                        "of the two HBM legs only)")
    p.add_argument("--calibration-copy-mib", type=int, default=256,
                   help="size of one untimed device-to-device copy whose HBM counters calibrate the traffic figure")
    p.add_argument("--next", action="store_true",
                   help="also measure the hybrid cache budget sweep and the recompute-vs-transfer sweep over evicted tokens")
    p.add_argument("--only", choices=["single_checkpoint", "sliding_window", "hybrid_budget", "evicted_tokens",
                                       "bounded_cache", "crossover", "workloads", "cpu_baselines"],
                   help="run only this one measurement and print its JSON (no headline line; for profiling its "
                        "kernels)")
    p.add_argument("--no-workloads", action="store_true",
                   help="skip the other configurations' steps (SmolLM fp32 layer, Qwen-1.5B shape, multi-turn)")
    p.add_argument("--all-turns", action="store_true", help="time all 20 turn boundaries of the multi-turn workload")
    return p.parse_args()


def op_timer(torch, np, default_iters):
    """op_time(fn, ...): average (or median) device time of fn() in us over iters calls, HIP
    events around each call, optionally after flush() (a cache-evicting write)."""
    def op_time(fn, iters=None, warm=2, flush=None, median=False):
        iters = iters or default_iters
        for _ in range(warm):
            fn()
        times = []
        for _ in range(iters):
            if flush is not None:
                flush()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            times.append((a, b))
        torch.cuda.synchronize()
        v = [a.elapsed_time(b) for a, b in times]
        return float(np.median(v) if median else np.mean(v)) * 1e3
    return op_time


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def source_hash():
    h = hashlib.sha256()
    for s in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2603_19664_amd", "csrc", s), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


class Call:
    """A libkvd entry point with its ctypes arguments built once (keeps host overhead per launch small)."""

    def __init__(self, fn, *args):
        self.fn, self.args = fn, args

    def __call__(self):
        st = self.fn(*self.args)
        if st != 0:
            from paper_2603_19664_amd import kvd
            raise kvd.KvdError(st, kvd.last_error())


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the library has no multi-GPU path (asked for --gpus {args.gpus}). "
              "The KV-Direct hot path shards over sequences, KV heads or keys with one exchange of split-K "
              "partials per layer; that exchange is not built.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2603_19664_amd import accounting as acc
    from paper_2603_19664_amd import configs, inputs
    from paper_2603_19664_amd import kvd

    torch.cuda.set_device(0)
    turns = tuple(range(1, 21)) if args.all_turns else (1, 5, 10, 15, 20)
    # one plain copy of known size (untimed): its FETCH_SIZE / WRITE_SIZE in a
    # counter run scale the measured kernels' counters to bytes
    if args.calibration_copy_mib > 0:
        src = torch.empty(args.calibration_copy_mib << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.only:
        op_time = op_timer(torch, np, 3)
        fn = {"single_checkpoint": lambda: run_single_checkpoint(torch, np, kvd, configs, inputs, log),
              "sliding_window": lambda: run_sliding(torch, kvd, configs, inputs, log),
              "hybrid_budget": lambda: run_hybrid(torch, np, kvd, configs, inputs, op_time, log),
              "evicted_tokens": lambda: run_evicted(torch, np, kvd, configs, inputs, op_time, log)[
                  "evicted_tokens"],
              "bounded_cache": lambda: run_bounded_cache(torch, np, kvd, configs, inputs, log),
              "crossover": lambda: run_crossover(args, torch, np, kvd, acc, configs, inputs, op_time, log),
              "workloads": lambda: run_workloads(args, torch, np, kvd, acc, configs, inputs, log, turns),
              "cpu_baselines": lambda: run_cpu_baselines(args, np, torch, configs, inputs, log)}[args.only]
        print(json.dumps({args.only: fn()}), flush=True)
        return
    dev = "cuda"
    wl = configs.GEMMA3_4B
    s = kvd.shape_of(wl).packed()   # weights in the packed MFMA layout (packed once, outside the step)
    sc = s.c()
    L, B, T = wl.layers, wl.batch, wl.ctx
    d, nq, nkv, hd = wl.d_model, wl.n_q, wl.n_kv, wl.head_dim
    lib = kvd.lib
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731

    log(f"[bench] workload {wl.name}: generating {L} layers of weights and residual checkpoints")
    layers = []
    for l in range(L):
        gamma, w_q, w_k, w_v = inputs.weights(wl, l, 0, dev)
        h, h_new = inputs.residuals(wl, l, B, T, 0, dev)
        layers.append(dict(gamma=gamma, w_q=kvd.kvd_pack_weights(s, w_q), w_k=kvd.kvd_pack_weights(s, w_k),
                           w_v=kvd.kvd_pack_weights(s, w_v), h=h, h_new=h_new, rw_k=w_k, rw_v=w_v, rw_q=w_q))
    pos0 = torch.zeros((B,), dtype=torch.int32, device=dev)
    pos_new = torch.full((B,), T, dtype=torch.int32, device=dev)
    q = torch.empty((B, nq, hd), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q)
    tk = torch.zeros((B, nkv, 1, hd), dtype=torch.bfloat16, device=dev)
    tv = torch.zeros_like(tk)
    tail = kvd.KvView(tk.data_ptr(), tv.data_ptr(), 1, 0)
    ws_f = kvd.workspace(s, kvd.KVD_OP_FUSED, B, T, 1)
    wsb_f = ws_f.numel()

    def calls_on(st):
        """The step's launches (per layer: project_qkv, fused) on stream st."""
        pj, fz = [], []
        for ly in layers:
            pj.append(Call(lib.kvd_project_qkv, ctypes.byref(sc), P(ly["h_new"]), P(ly["gamma"]), P(ly["w_q"]),
                           P(ly["w_k"]), P(ly["w_v"]), P(pos_new), B, P(q), ctypes.byref(tail), st))
            fz.append(Call(lib.kvd_fused_recompute_attn, ctypes.byref(sc), P(q), P(ly["h"]), T, P(ly["gamma"]),
                           P(ly["w_k"]), P(ly["w_v"]), P(pos0), B, T, ctypes.byref(tail), 1, P(out), P(ws_f), wsb_f,
                           None, st))
        return pj, fz

    proj, fused = calls_on(stream)

    def step(events=None, i=0, pj=proj, fz=fused):
        for l in range(L):
            pj[l]()
            if events is not None:
                events[i][l][0].record()
            fz[l]()
            if events is not None:
                events[i][l][1].record()

    # ---------------------------------------------------------------- timed region
    # value: the K timed steps are captured once as a HIP graph and replayed (the
    # same launches in the same order as eager steps; the replay is checked
    # bitwise against an eager step first).  The fused kernel's duration for the
    # roofline: HIP events around every fused launch over K eager steps on the
    # launch stream (events recorded inside a graph are not refreshed by replays,
    # and recorded eagerly they widen every kernel boundary by a few us, so the
    # two are measured in separate passes).
    K, W = args.steps, args.warmup
    log(f"[bench] warmup {W} steps")
    for _ in range(W):
        step()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        cst = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        gp, gf = calls_on(cst)
        for i in range(K):
            step(None, i, gp, gf)
    graph.replay()  # untimed: first launch of the graph
    torch.cuda.synchronize()
    out_graph = out.clone()
    step()
    torch.cuda.synchronize()
    if not torch.equal(out_graph.view(torch.int16), out.view(torch.int16)):
        raise RuntimeError("graph replay of the step differs from the eager step")
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"[bench] timing {K} steps (one graph replay)")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    t_start.record()
    graph.replay()
    t_end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = t_start.elapsed_time(t_end) / K
    del graph
    log(f"[bench] timing the fused kernel: {K} eager steps with events around each launch")
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(L)]
          for _ in range(K)]
    e_start, e_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e_start.record()
    for i in range(K):
        step(ev, i)
    e_end.record()
    torch.cuda.synchronize()
    ms_step_events = e_start.elapsed_time(e_end) / K
    fused_ms = float(np.mean([a.elapsed_time(b) for row in ev for (a, b) in row]))
    log(f"[bench] {ms_step:.3f} ms/step (wall {1e3 * wall / K:.3f}); with per-launch events "
        f"{ms_step_events:.3f} ms/step, fused kernel {1e3 * fused_ms:.1f} us/launch")

    flops = acc.fused_flops(B, T, 1, nq, nkv, d, hd)
    achieved = flops / (fused_ms * 1e-3) / 1e12
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if tr.get("source_hash") == source_hash() and tr.get("workload") == wl.name:
            traffic = tr.get("bytes_per_launch")

    # ---------------------------------------------------------------- per-op us/layer and baselines
    op_time = op_timer(torch, np, max(3, K))

    per_op = {}
    baselines = {}
    if not args.no_baselines:
        log("[bench] per-op timings (cycling the 34 layers)")
        cyc = lambda calls: (lambda c=[0]: (calls[c[0] % L](), c.__setitem__(0, c[0] + 1)))  # noqa: E731
        per_op["project_qkv_us"] = op_time(cyc(proj), iters=2 * L)
        per_op["fused_recompute_attn_us"] = op_time(cyc(fused), iters=2 * L)

        # cached-K/V baseline: a persistent bf16 cache per layer, prefilled once by the library
        log("[bench] cached-K/V baseline: prefilling 34 layers of bf16 K/V")
        S_c = kvd.kvd_num_splits(s, kvd.KVD_OP_CACHED_ATTN, B, T + 1)
        ws_c = kvd.workspace(s, kvd.KVD_OP_CACHED_ATTN, B, T + 1)
        cached, cproj = [], []
        caches = []
        for ly in layers:
            Kc = torch.empty((B, nkv, T + 1, hd), dtype=torch.bfloat16, device=dev)
            Vc = torch.empty_like(Kc)
            kvd.kvd_recompute_kv(s, ly["h"], ly["gamma"], ly["w_k"], ly["w_v"], pos0, T, Kc, Vc, 0)
            caches.append((Kc, Vc))
            vrow = kvd.KvView(Kc.data_ptr(), Vc.data_ptr(), T + 1, T)
            vall = kvd.KvView(Kc.data_ptr(), Vc.data_ptr(), T + 1, 0)
            caches.append((vrow, vall))
            cproj.append(Call(lib.kvd_project_qkv, ctypes.byref(sc), P(ly["h_new"]), P(ly["gamma"]), P(ly["w_q"]),
                              P(ly["w_k"]), P(ly["w_v"]), P(pos_new), B, P(q), ctypes.byref(vrow), stream))
            cached.append(Call(lib.kvd_cached_attn, ctypes.byref(sc), P(q), ctypes.byref(vall), B, T + 1, P(out),
                               P(ws_c), ws_c.numel(), stream))
        per_op["cached_attn_us"] = op_time(cyc(cached), iters=2 * L)
        # the 34 layers' cached attention back to back (no event between launches)
        b2b = _step_timer(torch, lambda: [c() for c in cached], steps=max(3, K // 2), warmup=2) / L
        per_op["cached_attn_us_back_to_back"] = 1e3 * b2b

        def cached_step():
            for l in range(L):
                cproj[l]()
                cached[l]()
        cached_ms = op_time(cached_step, iters=max(3, K // 2)) / 1e3
        baselines["cached_kv_ms_per_step"] = cached_ms
        baselines["cached_kv_tok_s"] = B / (cached_ms * 1e-3)
        cbytes = acc.cached_bytes(B, T + 1, nq, nkv, hd, 2, S_c)
        baselines["cached_attn_hbm_gbs"] = cbytes / (per_op["cached_attn_us"] * 1e-6) / 1e9
        baselines["cached_attn_hbm_frac"] = baselines["cached_attn_hbm_gbs"] / MI355X_HBM_PEAK_GBS
        baselines["cached_attn_hbm_gbs_back_to_back"] = cbytes / (b2b * 1e-3) / 1e9
        baselines["cached_attn_hbm_frac_back_to_back"] = baselines["cached_attn_hbm_gbs_back_to_back"] / \
            MI355X_HBM_PEAK_GBS
        baselines["cached_attn_splits"] = S_c

        # unfused recompute: recompute_kv writes K/V to HBM, decode_attn reads them back
        log("[bench] unfused recompute baseline")
        Ku = torch.empty((B, nkv, T + 1, hd), dtype=torch.bfloat16, device=dev)
        Vu = torch.empty_like(Ku)
        urow = kvd.KvView(Ku.data_ptr(), Vu.data_ptr(), T + 1, T)
        uall = kvd.KvView(Ku.data_ptr(), Vu.data_ptr(), T + 1, 0)
        uproj, urec, udec = [], [], []
        for ly in layers:
            uproj.append(Call(lib.kvd_project_qkv, ctypes.byref(sc), P(ly["h_new"]), P(ly["gamma"]), P(ly["w_q"]),
                              P(ly["w_k"]), P(ly["w_v"]), P(pos_new), B, P(q), ctypes.byref(urow), stream))
            urec.append(Call(lib.kvd_recompute_kv, ctypes.byref(sc), P(ly["h"]), T, P(ly["gamma"]), P(ly["w_k"]),
                             P(ly["w_v"]), P(pos0), B, T, ctypes.byref(uall), stream))
            udec.append(Call(lib.kvd_decode_attn, ctypes.byref(sc), P(q), ctypes.byref(uall), B, T + 1, P(out),
                             P(ws_c), ws_c.numel(), stream))
        per_op["recompute_kv_us"] = op_time(cyc(urec), iters=2 * L)
        per_op["decode_attn_us"] = op_time(cyc(udec), iters=2 * L)

        def unfused_step():
            for l in range(L):
                uproj[l]()
                urec[l]()
                udec[l]()
        unf_ms = op_time(unfused_step, iters=max(3, K // 2)) / 1e3
        baselines["unfused_ms_per_step"] = unf_ms
        baselines["unfused_tok_s"] = B / (unf_ms * 1e-3)
        rflops = acc.recompute_flops(B * T, nkv, d, hd)
        per_op["recompute_kv_tflops"] = rflops / (per_op["recompute_kv_us"] * 1e-6) / 1e12
        del caches

    # ---------------------------------------------------------------- crossover over batch size
    crossover = None
    if not args.no_crossover:
        crossover = run_crossover(args, torch, np, kvd, acc, configs, inputs, op_time, log)

    # ---------------------------------------------------------------- CPU oracle baseline
    cpu = None
    if not args.no_cpu_baseline:
        cpu = run_cpu_baseline(args, np, wl, layers, T, B, inputs, log)

    res = {
        "metric": "decode tok/s + µs/layer: recompute-K/V attn vs cached-KV read; MFMA% / HBM%",
        "value": B / (ms_step * 1e-3),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": ms_step,
        "us_per_layer": 1e3 * ms_step / L,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) residuals scaled per layer by U(0.5,4); random-init N(0,0.02) weights)",
        "config": {"workload": wl.name, "layers": L, "batch": B, "ctx": T, "keys_per_query": T + 1,
                   "d_model": d, "n_q_heads": nq, "n_kv_heads": nkv, "head_dim": hd,
                   "step": "per layer: kvd_project_qkv + kvd_fused_recompute_attn (split-K merge in-kernel)",
                   "launch": "the K timed steps captured once as a HIP graph and replayed"},
        "eager_ms_per_step_with_events": ms_step_events,
        "roofline": {"bound": "mfma", "kernel": "fused_kernel<bf16,256,64>", "achieved": achieved,
                     "peak": MI355X_BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": achieved / MI355X_BF16_PEAK_TFLOPS,
                     "traffic": traffic, "flops_per_launch": flops, "us_per_launch": 1e3 * fused_ms},
        "per_op_us": per_op,
        "baselines": baselines,
        "crossover": crossover,
        "cpu_baseline": cpu,
    }
    del layers
    torch.cuda.empty_cache()
    if not args.no_workloads:
        res["workloads"] = run_workloads(args, torch, np, kvd, acc, configs, inputs, log, turns)
    if not args.no_cpu_baseline:
        res["cpu_baselines"] = run_cpu_baselines(args, np, torch, configs, inputs, log)
    if args.next:
        res["next"] = run_next(args, torch, np, kvd, configs, inputs, op_time, log)
    print(json.dumps(res), flush=True)


def cold_flush(torch):
    """A 1 GiB read that evicts L2 and the 256 MB Infinity Cache before a timed op.  A read,
    not a write: a write flush leaves the Infinity Cache full of dirty lines, and their
    write-back during the timed op cost a pure-read kernel up to 40% of its bandwidth
    (measured on MI355X), which would flatter recompute against the cached read."""
    buf = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    return lambda: buf.sum()


def run_crossover(args, torch, np, kvd, acc, configs, inputs, op_time, log):
    """Fused recompute-attention vs cached-K/V attention (each with its split-K merge) for one
    Gemma-3-4B-shaped layer, context 2048 + current token, over batch size.  Each
    measurement runs after a cache-evicting read (cold_flush), so both sides read their
    inputs from HBM.  A third leg keeps the bf16 K/V cache in pinned host memory (a cache
    offloaded off the GPU): its K and V are copied over PCIe into HBM, then attended by the
    same cached-K/V kernel; the time is copy plus attention."""
    wl = configs.GEMMA3_SWEEP
    s = kvd.shape_of(wl).packed()
    T = wl.ctx
    flush = cold_flush(torch)
    rows = []
    for B in [int(x) for x in args.sweep_batches.split(",")]:
        log(f"[bench] crossover B={B}")
        gamma, w_q, w_k, w_v = (inputs.weights(wl, 0, 0, "cuda")[0],
                                *(kvd.kvd_pack_weights(s, w) for w in inputs.weights(wl, 0, 0, "cuda")[1:]))
        h, h_new = inputs.residuals(wl, 0, B, T, 0, "cuda")
        pos0 = torch.zeros((B,), dtype=torch.int32, device="cuda")
        pos_new = torch.full((B,), T, dtype=torch.int32, device="cuda")
        q = torch.empty((B, wl.n_q, wl.head_dim), dtype=torch.bfloat16, device="cuda")
        out = torch.empty_like(q)
        Kc = torch.empty((B, wl.n_kv, T + 1, wl.head_dim), dtype=torch.bfloat16, device="cuda")
        Vc = torch.empty_like(Kc)
        kvd.kvd_recompute_kv(s, h, gamma, w_k, w_v, pos0, T, Kc, Vc, 0)
        kvd.kvd_project_qkv(s, h_new, gamma, w_q, w_k, w_v, pos_new, q, Kc, Vc, T)
        tk, tv = Kc[:, :, T:T + 1].contiguous(), Vc[:, :, T:T + 1].contiguous()
        ws_f = kvd.workspace(s, kvd.KVD_OP_FUSED, B, T, 1)
        ws_c = kvd.workspace(s, kvd.KVD_OP_CACHED_ATTN, B, T + 1)
        fz = lambda: kvd.kvd_fused_recompute_attn(s, q, h, T, gamma, w_k, w_v, pos0, out, ws_f, tk, tv, 1)  # noqa
        cz = lambda: kvd.kvd_cached_attn(s, q, Kc, Vc, T + 1, out, ws_c)  # noqa: E731
        it = 10
        f_us = op_time(fz, iters=it, flush=flush, median=True)
        c_us = op_time(cz, iters=it, flush=flush, median=True)
        h_us = None
        if not args.no_host_cache:
            Kh = torch.empty(Kc.shape, dtype=Kc.dtype, pin_memory=True)
            Vh = torch.empty(Vc.shape, dtype=Vc.dtype, pin_memory=True)
            Kh.copy_(Kc)
            Vh.copy_(Vc)

            def hz():
                Kc.copy_(Kh, non_blocking=True)
                Vc.copy_(Vh, non_blocking=True)
                cz()
            h_us = op_time(hz, iters=5, flush=flush, median=True)
            del Kh, Vh
        kv_bytes = 2 * Kc.numel() * Kc.element_size()
        fl = acc.fused_flops(B, T, 1, wl.n_q, wl.n_kv, wl.d_model, wl.head_dim)
        S_c = kvd.kvd_num_splits(s, kvd.KVD_OP_CACHED_ATTN, B, T + 1)
        cb = acc.cached_bytes(B, T + 1, wl.n_q, wl.n_kv, wl.head_dim, 2, S_c)
        rows.append({"B": B, "fused_us": f_us, "cached_us": c_us, "ratio_fused_over_cached": f_us / c_us,
                     "fused_tflops": fl / (f_us * 1e-6) / 1e12,
                     "fused_mfma_frac": fl / (f_us * 1e-6) / 1e12 / MI355X_BF16_PEAK_TFLOPS,
                     "cached_gbs": cb / (c_us * 1e-6) / 1e9,
                     "cached_hbm_frac": cb / (c_us * 1e-6) / 1e9 / MI355X_HBM_PEAK_GBS, "cached_splits": S_c,
                     "host_cached_us": h_us, "ratio_fused_over_host_cached": None if h_us is None else f_us / h_us,
                     "host_copy_gbs": None if h_us is None else kv_bytes / ((h_us - c_us) * 1e-6) / 1e9})
        log(f"[bench] crossover B={B}: fused {f_us:.1f} us ({rows[-1]['fused_tflops']:.0f} TFLOP/s), cached "
            f"{c_us:.1f} us ({rows[-1]['cached_gbs']:.0f} GB/s)"
            + ("" if h_us is None else f", host-resident cache {h_us:.1f} us"))
        del h, Kc, Vc
        torch.cuda.empty_cache()
    faster = [r["B"] for r in rows if r["ratio_fused_over_cached"] < 1.0]
    faster_host = [r["B"] for r in rows
                   if r["ratio_fused_over_host_cached"] is not None and r["ratio_fused_over_host_cached"] < 1.0]
    return {"workload": wl.name, "ctx": T, "rows": rows, "batches_where_recompute_wins": faster,
            "batches_where_recompute_beats_host_cache": faster_host,
            "note": "medians of 10 calls (5 for the host-resident cache), each after a 1 GiB cache-evicting read; "
                    "every leg includes its split-K merge; host_copy_gbs = K/V bytes / (host-resident time - "
                    "cached time)"}


def run_next(args, torch, np, kvd, configs, inputs, op_time, log):
    """Two measurements on one Gemma-3-4B-shaped layer (context 4096 + the current token),
    each op timed with HIP events after a cache-evicting read (cold_flush):

    hybrid_budget: Algorithm 1 with a cache budget of W tokens.  The W most recent context
      tokens keep stored bf16 K/V and form the fused kernel's tail with the current token;
      the older T - W are recomputed from their checkpoints in the kernel.  Every token keeps
      its checkpoint (STORE_RESIDUAL), so memory = checkpoints of T tokens + K/V of W + 1.
      The per-token costs are the slopes of the fused time in the recomputed and the stored
      token counts.

    evicted_tokens: N evicted tokens' K/V made available again, three ways: recomputed from
      their checkpoints (kvd_recompute_kv), copied from a bf16 copy in HBM, and copied from a
      bf16 copy in pinned host memory over PCIe (token-major, so each is one contiguous copy).
      Medians of 11 calls (a PCIe copy occasionally takes far longer)."""
    res = {"hybrid_budget": run_hybrid(torch, np, kvd, configs, inputs, op_time, log),
           "bounded_cache": run_bounded_cache(torch, np, kvd, configs, inputs, log)}
    res.update(run_evicted(torch, np, kvd, configs, inputs, op_time, log))
    res["sliding_window"] = run_sliding(torch, kvd, configs, inputs, log)
    res["single_checkpoint"] = run_single_checkpoint(torch, np, kvd, configs, inputs, log)
    return res


def _next_setup(torch, kvd, configs, inputs):
    wl = configs.GEMMA3_4B
    s = kvd.shape_of(wl).packed()
    flush = cold_flush(torch)
    gamma, w_q, w_k, w_v = inputs.weights(wl, 0, 0, "cuda")
    w_q, w_k, w_v = (kvd.kvd_pack_weights(s, w) for w in (w_q, w_k, w_v))
    return wl, s, flush, gamma, w_q, w_k, w_v


def run_hybrid(torch, np, kvd, configs, inputs, op_time, log):
    """The hybrid cache budget sweep (see run_next)."""
    wl, s, flush, gamma, w_q, w_k, w_v = _next_setup(torch, kvd, configs, inputs)
    T, d, nkv, hd = wl.ctx, wl.d_model, wl.n_kv, wl.head_dim
    rows = []
    for B in (1, 8):
        log(f"[bench] next: hybrid budget B={B}")
        h, h_new = inputs.residuals(wl, 0, B, T, 0, "cuda")
        pos0 = torch.zeros((B,), dtype=torch.int32, device="cuda")
        pos_new = torch.full((B,), T, dtype=torch.int32, device="cuda")
        q = torch.empty((B, wl.n_q, hd), dtype=torch.bfloat16, device="cuda")
        out = torch.empty_like(q)
        Kc = torch.empty((B, nkv, T + 1, hd), dtype=torch.bfloat16, device="cuda")
        Vc = torch.empty_like(Kc)
        kvd.kvd_recompute_kv(s, h, gamma, w_k, w_v, pos0, T, Kc, Vc, 0)
        kvd.kvd_project_qkv(s, h_new, gamma, w_q, w_k, w_v, pos_new, q, Kc, Vc, T)
        for W in (0, 256, 1024, 2048, 3072, 4096):
            T_rec, T_tail = T - W, W + 1
            ws = kvd.workspace(s, kvd.KVD_OP_FUSED, B, T_rec, T_tail)
            fz = lambda: kvd.kvd_fused_recompute_attn(s, q, h, T_rec, gamma, w_k, w_v, pos0, out, ws,  # noqa: E731
                                                     Kc, Vc, T_tail, T_rec)
            us = op_time(fz, iters=10, flush=flush)
            rows.append({"B": B, "budget_tokens": W, "recomputed_tokens": T_rec, "stored_rows": T_tail,
                         "fused_us": us, "checkpoint_bytes": B * T * d * 2,
                         "kv_bytes": B * T_tail * 2 * nkv * hd * 2})
            del ws
        del h, h_new, Kc, Vc
        torch.cuda.empty_cache()
    slopes = {}
    for B in (1, 8):
        r = [x for x in rows if x["B"] == B]
        W = np.array([x["budget_tokens"] for x in r], dtype=np.float64)
        t = np.array([x["fused_us"] for x in r])
        a, b = np.polyfit(W, t, 1)[::-1]  # t ~ a + b W
        read_per_token = r[-1]["fused_us"] / (T + 1)  # W = T: every key is read
        slopes[str(B)] = {"us_per_recomputed_minus_stored_token": -b, "fit_intercept_us": a,
                          "us_per_stored_token_read": read_per_token,
                          "us_per_recomputed_token": read_per_token - b}
    return {"workload": "gemma3-4b layer, ctx 4096 + current token", "rows": rows, "per_token_costs": slopes}


def run_bounded_cache(torch, np, kvd, configs, inputs, log, steps=300, budgets=(0, 64, 256, 1024), start=4096):
    """Algorithm 1's bounded cache in a decode loop (paper_2603_19664_amd.budget.BoundedCache):
    one Gemma-3-4B-shaped layer, B = 1 and 8, a history of `start` tokens (the last `budget`
    of them in the cache ring, the rest evicted to checkpoints), then `steps` decode steps
    (STORE_RESIDUAL, Q/K_t/V_t into the ring, fused recompute + attention, eviction).  Reports
    the device time per step (HIP events around the loop; the three launches of a step are
    issued from Python) and the fused call's own time, and the memory per layer and sequence
    against Eq. total_mem."""
    from paper_2603_19664_amd.budget import BoundedCache
    wl = configs.GEMMA3_4B
    s = kvd.shape_of(wl).packed()
    gamma, w_q, w_k, w_v = inputs.weights(wl, 0, 0, "cuda")
    w_q, w_k, w_v = (kvd.kvd_pack_weights(s, w) for w in (w_q, w_k, w_v))
    rows = []
    for B in (1, 8):
        h_all, _ = inputs.residuals(wl, 0, B, start + steps, 0, "cuda")
        pos0 = torch.zeros((B,), dtype=torch.int32, device="cuda")
        for budget in budgets:
            log(f"[bench] next: bounded cache B={B} budget={budget}")
            cache = BoundedCache(s, B, budget, start + steps, pos0)
            st = cache.state
            cache.ckpt[:, :start].copy_(h_all[:, :start])           # the history's checkpoints
            st.T, st.T_rec, st.head, st.n_cached = start, start - budget, 0, budget
            if budget > 0:                                          # the cached tokens' K/V, ring slots 0..budget-1
                kvd.kvd_recompute_kv(s, h_all[:, start - budget:start].contiguous(), gamma, w_k, w_v,
                                     (pos0 + start - budget).to(torch.int32), budget, cache.ring_k, cache.ring_v, 0)
            out = torch.empty((B, s.n_q_heads, s.head_dim), dtype=torch.bfloat16, device="cuda")
            h_steps = [h_all[:, start + i].contiguous() for i in range(steps)]
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for i in range(steps):
                cache.step(h_steps[i], gamma, w_q, w_k, w_v, out)
            b.record()
            torch.cuda.synchronize()
            step_us = a.elapsed_time(b) * 1e3 / steps
            # the fused call alone at the final state's shape
            ws = cache.ws
            fz = lambda: kvd.kvd_fused_recompute_attn(s, cache.q, cache.ckpt, st.T_rec, gamma, w_k, w_v, pos0, out,  # noqa
                                                     ws, cache.ring_k, cache.ring_v, st.n_cached + 1, st.head)
            for _ in range(3):
                fz()
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(20)]
            for e0, e1 in ev:
                e0.record()
                fz()
                e1.record()
            torch.cuda.synchronize()
            fused_us = float(np.median([e0.elapsed_time(e1) for e0, e1 in ev])) * 1e3
            m = st.memory_bytes(s.d_model, s.n_kv_heads, s.head_dim, 2)
            rows.append({"B": B, "budget": budget, "tokens_after": st.T, "recomputed": st.T_rec,
                         "cached": st.n_cached, "us_per_step_loop": step_us, "fused_us": fused_us,
                         "memory_per_layer_seq": m})
            log(f"[bench] next: bounded cache B={B} budget={budget}: {step_us:.1f} us/step, fused {fused_us:.1f} us")
            del cache
        del h_all
        torch.cuda.empty_cache()
    return {"workload": f"gemma3-4b layer, {start} tokens of history then {steps} decode steps", "rows": rows}


def run_evicted(torch, np, kvd, configs, inputs, op_time, log):
    """Recompute vs copy of N evicted tokens' K/V (see run_next)."""
    wl, s, flush, gamma, w_q, w_k, w_v = _next_setup(torch, kvd, configs, inputs)
    T, nkv, hd = wl.ctx, wl.n_kv, wl.head_dim
    res = {}
    log("[bench] next: evicted tokens, recompute vs HBM copy vs host copy")
    B = 1
    h, _ = inputs.residuals(wl, 0, B, T, 0, "cuda")
    pos0 = torch.zeros((B,), dtype=torch.int32, device="cuda")
    Kc = torch.empty((B, nkv, T, hd), dtype=torch.bfloat16, device="cuda")
    Vc = torch.empty_like(Kc)
    kvd.kvd_recompute_kv(s, h, gamma, w_k, w_v, pos0, T, Kc, Vc, 0)
    kv_dev = torch.stack([Kc[0].transpose(0, 1), Vc[0].transpose(0, 1)], dim=1).contiguous()  # [T][2][n_kv][hd]
    kv_host = torch.empty(kv_dev.shape, dtype=kv_dev.dtype, pin_memory=True)
    kv_host.copy_(kv_dev)
    erows = []
    for N in (1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096):
        Kr = torch.empty((B, nkv, N, hd), dtype=torch.bfloat16, device="cuda")
        Vr = torch.empty_like(Kr)
        dst = torch.empty((N,) + tuple(kv_dev.shape[1:]), dtype=kv_dev.dtype, device="cuda")
        rec = lambda: kvd.kvd_recompute_kv(s, h, gamma, w_k, w_v, pos0, N, Kr, Vr, 0)  # noqa: E731
        hbm = lambda: dst.copy_(kv_dev[:N])  # noqa: E731
        host = lambda: dst.copy_(kv_host[:N], non_blocking=True)  # noqa: E731
        e = {"N": N, "kv_bytes": N * 2 * nkv * hd * 2,
             "recompute_us": op_time(rec, iters=11, flush=flush, median=True),
             "hbm_copy_us": op_time(hbm, iters=11, flush=flush, median=True),
             "host_copy_us": op_time(host, iters=11, flush=flush, median=True)}
        erows.append(e)
        log(f"[bench] next: N={N}: recompute {e['recompute_us']:.1f} us, HBM copy {e['hbm_copy_us']:.1f} us, "
            f"host copy {e['host_copy_us']:.1f} us")
    res["evicted_tokens"] = {
        "workload": "gemma3-4b layer, B=1; K/V of N evicted tokens (N * 4 KiB)", "rows": erows,
        "recompute_faster_than_hbm_copy": [e["N"] for e in erows if e["recompute_us"] < e["hbm_copy_us"]],
        "recompute_faster_than_host_copy": [e["N"] for e in erows if e["recompute_us"] < e["host_copy_us"]]}
    del h, Kc, Vc, kv_dev, kv_host, flush
    torch.cuda.empty_cache()
    return res


def block_flops(B, T, d, n_q, n_kv, hd, d_ff):
    """Algorithmic flops of one pre-norm block over B sequences of T positions: the
    Q/K/V, W_o and MLP products plus causal attention (scores and weighted sum over
    t + 1 keys at position t)."""
    proj = 2 * B * T * d * (n_q + 2 * n_kv) * hd + 2 * B * T * n_q * hd * d + 2 * B * T * 3 * d * d_ff
    attn = 4 * B * n_q * hd * (T * (T + 1) // 2)
    return proj + attn


def run_single_checkpoint(torch, np, kvd, configs, inputs, log, d_ff=10240, n_distinct=4):
    """The single-checkpoint scheme (one residual per token for all layers): recomputing
    h^(l) means running blocks 0 .. l-1 over every position (kvd_block_forward).  A
    Gemma-3-4B-shaped block (d 2560, 8 q / 4 KV heads of 256; d_ff 10240 is a stand-in,
    the paper does not give the MLP width), B = 1, T = 1024 and 4096: one block's time,
    and the 34 blocks that recompute every layer's residuals once (n_distinct layers of
    weights cycled), HIP events around the calls."""
    wl = configs.GEMMA3_4B
    s = kvd.shape_of(wl).packed()
    L, d, nq, nkv, hd = wl.layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim
    blocks = []
    for l in range(n_distinct):
        gamma, w_q, w_k, w_v = inputs.weights(wl, l, 0, "cuda")
        w_o, gamma_mlp, w_gate, w_up, w_down = inputs.block_weights(wl, l, d_ff, 0, "cuda")
        pw = lambda w: kvd.kvd_pack_weights(s, w)  # noqa: E731
        lw = (gamma, pw(w_q), pw(w_k), pw(w_v), kvd.kvd_pack_matrix(w_o), gamma_mlp, pw(w_gate), pw(w_up),
              kvd.kvd_pack_matrix(w_down))
        del w_q, w_k, w_v, w_o, w_gate, w_up, w_down
        blocks.append((lw, kvd.block_weights(*lw)))
    rows = []
    for T in (1024, 4096):
        B = 1
        log(f"[bench] next: single checkpoint, block forward T={T}")
        h, _ = inputs.residuals(wl, 0, B, T, 0, "cuda")
        h = h.contiguous()
        bufs = [h, torch.empty_like(h)]
        pos0 = torch.zeros((B,), dtype=torch.int32, device="cuda")
        ws = torch.empty(kvd.kvd_block_workspace_bytes(s, d_ff, B, T), dtype=torch.uint8, device="cuda")
        sc = s.c()
        P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
        st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        calls = [Call(kvd.lib.kvd_block_forward, ctypes.byref(sc), ctypes.byref(blocks[i % n_distinct][1]),
                      P(bufs[i % 2]), P(bufs[(i + 1) % 2]), P(pos0), B, T, P(ws), ws.numel(), st)
                 for i in range(L)]
        one = _step_timer(torch, calls[0], steps=10, warmup=2)
        # the recompute of all L layers' residuals: L blocks in a row (ping-pong buffers)
        full = _step_timer(torch, lambda: [c() for c in calls], steps=3, warmup=1)
        fl = block_flops(B, T, d, nq, nkv, hd, d_ff)
        rows.append({"B": B, "T": T, "block_ms": one, "block_tflops": fl / (one * 1e-3) / 1e12,
                     "all_layers_ms": full, "all_layers_tflops": L * fl / (full * 1e-3) / 1e12,
                     "single_checkpoint_bytes": B * T * d * 2, "per_layer_checkpoint_bytes": L * B * T * d * 2,
                     "kv_cache_bytes": L * B * T * 2 * nkv * hd * 2})
        log(f"[bench] next: single checkpoint T={T}: block {one:.3f} ms ({rows[-1]['block_tflops']:.0f} TFLOP/s), "
            f"{L} blocks {full:.2f} ms")
        del h, bufs, ws
        torch.cuda.empty_cache()
    del blocks
    torch.cuda.empty_cache()
    return {"workload": f"gemma3-4b-shaped block (d_ff {d_ff}), {L} layers, B=1", "rows": rows}


def run_sliding(torch, kvd, configs, inputs, log, window=1024):
    """Sliding-window layers: a Gemma-3-4B-shaped decode step (34 layers, context 4096 + the
    current token) whose layers l with l % 6 != 5 are sliding-window layers (29 of 34; the
    window is a stand-in, the paper does not give its size) against the all-global step on
    the same inputs, for B = 1 and 8.  Recompute path: kvd_project_qkv (the current token at
    its window index on sliding layers) + kvd_fused_window_attn, which recomputes only the
    window's residual rows.  Cached path: kvd_project_qkv into the cache + kvd_cached_attn
    over all T + 1 rows (global layers) or over a window-sized buffer (sliding layers).
    Eager steps of prebuilt C-ABI calls; HIP events around 10 steps after 2 warm-up steps."""
    wl = configs.GEMMA3_4B
    s = kvd.shape_of(wl).packed()
    sc = s.c()
    L, T, nq, nkv, hd = wl.layers, wl.ctx, wl.n_q, wl.n_kv, wl.head_dim
    lib, dev = kvd.lib, "cuda"
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    sliding = [l % 6 != 5 for l in range(L)]
    W = window
    rows = []
    for B in (1, 8):
        log(f"[bench] next: sliding-window layers, B={B}")
        layers = _model_layers(wl, s, kvd, inputs, L, B, T, dev)
        pos0 = torch.zeros((B,), dtype=torch.int32, device=dev)
        pos_g = torch.full((B,), T, dtype=torch.int32, device=dev)
        pos_w = torch.full((B,), W - 1, dtype=torch.int32, device=dev)
        q = torch.empty((B, nq, hd), dtype=torch.bfloat16, device=dev)
        out = torch.empty_like(q)
        tk = torch.zeros((B, nkv, 1, hd), dtype=torch.bfloat16, device=dev)
        tv = torch.zeros_like(tk)
        tail = kvd.KvView(tk.data_ptr(), tv.data_ptr(), 1, 0)
        ws = kvd.workspace(s, kvd.KVD_OP_FUSED, B, T, 1)   # suffices for every call below

        def fused_step(use_window):
            calls = []
            for ly, sw in zip(layers, sliding):
                sw = sw and use_window
                calls.append(Call(lib.kvd_project_qkv, ctypes.byref(sc), P(ly["h_new"]), P(ly["gamma"]),
                                  P(ly["w_q"]), P(ly["w_k"]), P(ly["w_v"]), P(pos_w if sw else pos_g), B, P(q),
                                  ctypes.byref(tail), stream))
                if sw:
                    calls.append(Call(lib.kvd_fused_window_attn, ctypes.byref(sc), P(q), P(ly["h"]), T,
                                      P(ly["gamma"]), P(ly["w_k"]), P(ly["w_v"]), B, T, ctypes.byref(tail), 1, W,
                                      P(out), P(ws), ws.numel(), stream))
                else:
                    calls.append(Call(lib.kvd_fused_recompute_attn, ctypes.byref(sc), P(q), P(ly["h"]), T,
                                      P(ly["gamma"]), P(ly["w_k"]), P(ly["w_v"]), P(pos0), B, T,
                                      ctypes.byref(tail), 1, P(out), P(ws), ws.numel(), None, stream))
            return lambda: [c() for c in calls]

        ms_fg = _step_timer(torch, fused_step(False), steps=10, warmup=2)
        ms_fw = _step_timer(torch, fused_step(True), steps=10, warmup=2)
        # cached: a full (T + 1)-row cache per global layer, a W-row buffer per sliding layer
        wsc = kvd.workspace(s, kvd.KVD_OP_CACHED_ATTN, B, T + 1)
        caches = []
        for ly, sw in zip(layers, sliding):
            Kc = torch.empty((B, nkv, T + 1, hd), dtype=torch.bfloat16, device=dev)
            Vc = torch.empty_like(Kc)
            kvd.kvd_recompute_kv(s, ly["h"], ly["gamma"], ly["w_k"], ly["w_v"], pos0, T, Kc, Vc, 0)
            caches.append((Kc, Vc, kvd.KvView(Kc.data_ptr(), Vc.data_ptr(), T + 1, T),
                           kvd.KvView(Kc.data_ptr(), Vc.data_ptr(), T + 1, 0),
                           kvd.KvView(Kc.data_ptr(), Vc.data_ptr(), T + 1, T + 1 - W)))

        def cached_step(use_window):
            calls = []
            for ly, sw, (_, _, vrow, vall, vwin) in zip(layers, sliding, caches):
                sw = sw and use_window
                calls.append(Call(lib.kvd_project_qkv, ctypes.byref(sc), P(ly["h_new"]), P(ly["gamma"]),
                                  P(ly["w_q"]), P(ly["w_k"]), P(ly["w_v"]), P(pos_g), B, P(q),
                                  ctypes.byref(vrow), stream))
                calls.append(Call(lib.kvd_cached_attn, ctypes.byref(sc), P(q), ctypes.byref(vwin if sw else vall),
                                  B, W if sw else T + 1, P(out), P(wsc), wsc.numel(), stream))
            return lambda: [c() for c in calls]

        ms_cg = _step_timer(torch, cached_step(False), steps=10, warmup=2)
        ms_cw = _step_timer(torch, cached_step(True), steps=10, warmup=2)
        rows.append({"B": B, "fused_all_global_ms": ms_fg, "fused_sliding_ms": ms_fw,
                     "cached_all_global_ms": ms_cg, "cached_sliding_ms": ms_cw,
                     "fused_sliding_tok_s": B / (ms_fw * 1e-3), "cached_sliding_tok_s": B / (ms_cw * 1e-3)})
        log(f"[bench] next: sliding B={B}: fused {ms_fg:.3f} -> {ms_fw:.3f} ms/step, "
            f"cached {ms_cg:.3f} -> {ms_cw:.3f} ms/step")
        del layers, caches, ws, wsc
        torch.cuda.empty_cache()
    return {"workload": "gemma3-4b, 34 layers, ctx 4096 + current token", "window": W,
            "sliding_layers": int(sum(sliding)), "global_layers": [l for l in range(L) if not sliding[l]],
            "rows": rows}


def _step_timer(torch, step, steps, warmup):
    """ms per call of step(), HIP events around `steps` back-to-back calls after `warmup`."""
    for _ in range(warmup):
        step()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(steps):
        step()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / steps


def _model_layers(wl, s, kvd, inputs, L, B, T_cap, dev, packed=True):
    layers = []
    pk = (lambda w: kvd.kvd_pack_weights(s, w)) if packed else (lambda w: w)  # noqa: E731
    for l in range(L):
        gamma, w_q, w_k, w_v = inputs.weights(wl, l, 0, dev)
        h, h_new = inputs.residuals(wl, l, B, T_cap, 0, dev)
        layers.append(dict(gamma=gamma, w_q=pk(w_q), w_k=pk(w_k), w_v=pk(w_v), h=h, h_new=h_new))
        del w_q, w_k, w_v
    return layers


def run_workloads(args, torch, np, kvd, acc, configs, inputs, log, turns=(1, 5, 10, 15, 20), c4_steps=10):
    """The other configurations' decode steps, through the same C ABI calls as the headline
    step (per layer: kvd_project_qkv, then kvd_fused_recompute_attn with the current token as
    a one-row tail and the split-K merge in-kernel), HIP events around back-to-back steps:

      smollm_fp32: one SmolLM2-135M-shaped layer in fp32, 256 context tokens (the parity config);
      qwen_1_5b:   28 Qwen2.5-1.5B-shaped layers, B = 8, 16384 context tokens at per-sequence
                   position offsets, fused step against the cached-K/V step on the same inputs;
      multiturn:   34 Gemma-3-4B-shaped layers, B = 16, a decode step at turn boundaries of the
                   20 x 256-token conversation (checkpoints only; the cached step at turn 20 for
                   comparison), with the HBM footprint of each scheme."""
    lib, dev = kvd.lib, "cuda"
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    res = {}

    def fused_calls(sc, layers, B, T, h_ld, pos0, pos_new, q, out, tail, ws):
        calls = []
        for ly in layers:
            calls.append(Call(lib.kvd_project_qkv, ctypes.byref(sc), P(ly["h_new"]), P(ly["gamma"]), P(ly["w_q"]),
                              P(ly["w_k"]), P(ly["w_v"]), P(pos_new), B, P(q), ctypes.byref(tail), stream))
            calls.append(Call(lib.kvd_fused_recompute_attn, ctypes.byref(sc), P(q), P(ly["h"]), h_ld,
                              P(ly["gamma"]), P(ly["w_k"]), P(ly["w_v"]), P(pos0), B, T, ctypes.byref(tail), 1,
                              P(out), P(ws), ws.numel(), None, stream))
        return calls

    def cached_calls(sc, layers, caches, B, T, pos_new, q, out, wsc):
        calls = []
        for ly, (Kc, Vc, vrow, vall) in zip(layers, caches):
            calls.append(Call(lib.kvd_project_qkv, ctypes.byref(sc), P(ly["h_new"]), P(ly["gamma"]), P(ly["w_q"]),
                              P(ly["w_k"]), P(ly["w_v"]), P(pos_new), B, P(q), ctypes.byref(vrow), stream))
            calls.append(Call(lib.kvd_cached_attn, ctypes.byref(sc), P(q), ctypes.byref(vall), B, T + 1, P(out),
                              P(wsc), wsc.numel(), stream))
        return calls

    def prefill(s, layers, B, T, pos0):
        caches = []
        for ly in layers:
            Kc = torch.empty((B, s.n_kv_heads, T + 1, s.head_dim), dtype=torch.bfloat16, device=dev)
            Vc = torch.empty_like(Kc)
            kvd.kvd_recompute_kv(s, ly["h"], ly["gamma"], ly["w_k"], ly["w_v"], pos0, T, Kc, Vc, 0)
            caches.append((Kc, Vc, kvd.KvView(Kc.data_ptr(), Vc.data_ptr(), T + 1, T),
                           kvd.KvView(Kc.data_ptr(), Vc.data_ptr(), T + 1, 0)))
        return caches

    # ---- SmolLM2-135M layer, fp32 (the parity config): one decode step
    wl = configs.SMOLLM_FP32
    s = kvd.shape_of(wl)
    sc = s.c()
    B, T = wl.batch, wl.ctx
    log(f"[bench] workloads: {wl.name}")
    layers = _model_layers(wl, s, kvd, inputs, 1, B, T, dev, packed=False)
    pos0 = torch.zeros((B,), dtype=torch.int32, device=dev)
    pos_new = torch.full((B,), T, dtype=torch.int32, device=dev)
    q = torch.empty((B, wl.n_q, wl.head_dim), dtype=torch.float32, device=dev)
    out = torch.empty_like(q)
    tk = torch.zeros((B, wl.n_kv, 1, wl.head_dim), dtype=torch.float32, device=dev)
    tv = torch.zeros_like(tk)
    tail = kvd.KvView(tk.data_ptr(), tv.data_ptr(), 1, 0)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, B, T, 1)
    calls = fused_calls(sc, layers, B, T, T, pos0, pos_new, q, out, tail, ws)
    ms = _step_timer(torch, lambda: [c() for c in calls], steps=50, warmup=5)
    res["smollm_fp32"] = {"workload": wl.name, "layers": 1, "batch": B, "ctx": T, "dtype": "f32",
                          "us_per_layer": 1e3 * ms, "tok_s": B / (ms * 1e-3),
                          "note": "the parity config: fp32 on the vector ALUs (no fp32 MFMA path), 12 workgroups "
                                  "of 64 keys; latency bound"}
    del layers, calls
    torch.cuda.empty_cache()

    # ---- Qwen-1.5B shape: 28 layers, B = 8, 16384 checkpointed tokens + current token
    wl = configs.QWEN_1_5B
    s = kvd.shape_of(wl).packed()
    sc = s.c()
    L, B, T = wl.layers, wl.batch, wl.ctx
    log(f"[bench] workloads: {wl.name}: generating {L} layers")
    layers = _model_layers(wl, s, kvd, inputs, L, B, T, dev)
    pos0 = inputs.positions(wl, B).to(dev)
    pos_new = (pos0 + T).to(torch.int32)
    q = torch.empty((B, wl.n_q, wl.head_dim), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q)
    tk = torch.zeros((B, wl.n_kv, 1, wl.head_dim), dtype=torch.bfloat16, device=dev)
    tv = torch.zeros_like(tk)
    tail = kvd.KvView(tk.data_ptr(), tv.data_ptr(), 1, 0)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, B, T, 1)
    calls = fused_calls(sc, layers, B, T, T, pos0, pos_new, q, out, tail, ws)
    ms = _step_timer(torch, lambda: [c() for c in calls], steps=c4_steps, warmup=2)
    flops = L * acc.fused_flops(B, T, 1, wl.n_q, wl.n_kv, wl.d_model, wl.head_dim)
    entry = {"workload": wl.name, "layers": L, "batch": B, "ctx": T, "ms_per_step": ms, "tok_s": B / (ms * 1e-3),
             "us_per_layer": 1e3 * ms / L, "fused_path_tflops": flops / (ms * 1e-3) / 1e12,
             "fused_path_mfma_frac": flops / (ms * 1e-3) / 1e12 / MI355X_BF16_PEAK_TFLOPS}
    log(f"[bench] workloads: {wl.name}: fused step {ms:.3f} ms")
    caches = prefill(s, layers, B, T, pos0)
    wsc = kvd.workspace(s, kvd.KVD_OP_CACHED_ATTN, B, T + 1)
    ccalls = cached_calls(sc, layers, caches, B, T, pos_new, q, out, wsc)
    cms = _step_timer(torch, lambda: [c() for c in ccalls], steps=c4_steps, warmup=2)
    catt = _step_timer(torch, lambda: [c() for c in ccalls[1::2]], steps=c4_steps, warmup=2)
    cbytes = L * acc.cached_bytes(B, T + 1, wl.n_q, wl.n_kv, wl.head_dim, 2,
                                  kvd.kvd_num_splits(s, kvd.KVD_OP_CACHED_ATTN, B, T + 1))
    entry.update({"cached_ms_per_step": cms, "cached_tok_s": B / (cms * 1e-3),
                  "cached_attn_us_per_layer": 1e3 * catt / L, "cached_attn_gbs": cbytes / (catt * 1e-3) / 1e9,
                  "cached_attn_hbm_frac": cbytes / (catt * 1e-3) / 1e9 / MI355X_HBM_PEAK_GBS,
                  "checkpoint_bytes": L * B * T * wl.d_model * 2,
                  "kv_cache_bytes": L * B * (T + 1) * 2 * wl.n_kv * wl.head_dim * 2})
    log(f"[bench] workloads: {wl.name}: cached step {cms:.3f} ms (attention {catt:.3f} ms)")
    res["qwen_1_5b"] = entry
    del layers, caches, calls, ccalls
    torch.cuda.empty_cache()

    # ---- multi-turn conversation: Gemma 3-4B shape, 34 layers, B = 16, 20 turns of 256 tokens
    wl = configs.GEMMA3_MULTITURN
    s = kvd.shape_of(wl).packed()
    sc = s.c()
    L, B, Tmax = wl.layers, wl.batch, wl.turns * wl.turn_tokens
    log(f"[bench] workloads: {wl.name}: generating {L} layers of {Tmax}-token checkpoints")
    layers = _model_layers(wl, s, kvd, inputs, L, B, Tmax, dev)
    pos0 = torch.zeros((B,), dtype=torch.int32, device=dev)
    q = torch.empty((B, wl.n_q, wl.head_dim), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q)
    tk = torch.zeros((B, wl.n_kv, 1, wl.head_dim), dtype=torch.bfloat16, device=dev)
    tv = torch.zeros_like(tk)
    tail = kvd.KvView(tk.data_ptr(), tv.data_ptr(), 1, 0)
    rows = []
    for k in turns:
        T = k * wl.turn_tokens
        pos_new = torch.full((B,), T, dtype=torch.int32, device=dev)
        ws = kvd.workspace(s, kvd.KVD_OP_FUSED, B, T, 1)
        calls = fused_calls(sc, layers, B, T, Tmax, pos0, pos_new, q, out, tail, ws)
        ms = _step_timer(torch, lambda: [c() for c in calls], steps=3, warmup=1)
        flops = L * acc.fused_flops(B, T, 1, wl.n_q, wl.n_kv, wl.d_model, wl.head_dim)
        rows.append({"turn": k, "ctx": T, "ms_per_step": ms, "tok_s": B / (ms * 1e-3), "us_per_layer": 1e3 * ms / L,
                     "fused_path_tflops": flops / (ms * 1e-3) / 1e12,
                     "fused_path_mfma_frac": flops / (ms * 1e-3) / 1e12 / MI355X_BF16_PEAK_TFLOPS,
                     "checkpoint_bytes": L * B * T * wl.d_model * 2,
                     "kv_cache_equiv_bytes": L * B * T * 2 * wl.n_kv * wl.head_dim * 2,
                     "single_checkpoint_bytes": B * T * wl.d_model * 2, "workspace_bytes": ws.numel()})
        log(f"[bench] workloads: turn {k} ctx {T}: {ms:.3f} ms/step")
    entry = {"workload": wl.name, "layers": L, "batch": B, "turn_tokens": wl.turn_tokens, "turns": rows}
    # the cached-K/V step at the last turn on the same inputs (per-layer prefilled caches)
    T = Tmax
    pos_new = torch.full((B,), T, dtype=torch.int32, device=dev)
    caches = prefill(s, layers, B, T, pos0)
    wsc = kvd.workspace(s, kvd.KVD_OP_CACHED_ATTN, B, T + 1)
    ccalls = cached_calls(sc, layers, caches, B, T, pos_new, q, out, wsc)
    cms = _step_timer(torch, lambda: [c() for c in ccalls], steps=3, warmup=1)
    catt = _step_timer(torch, lambda: [c() for c in ccalls[1::2]], steps=3, warmup=1)
    cbytes = L * acc.cached_bytes(B, T + 1, wl.n_q, wl.n_kv, wl.head_dim, 2,
                                  kvd.kvd_num_splits(s, kvd.KVD_OP_CACHED_ATTN, B, T + 1))
    entry["cached_last_turn"] = {"ctx": T, "ms_per_step": cms, "tok_s": B / (cms * 1e-3),
                                 "attn_us_per_layer": 1e3 * catt / L, "attn_gbs": cbytes / (catt * 1e-3) / 1e9,
                                 "attn_hbm_frac": cbytes / (catt * 1e-3) / 1e9 / MI355X_HBM_PEAK_GBS}
    log(f"[bench] workloads: cached step at turn {wl.turns}: {cms:.3f} ms (attention {catt:.3f} ms)")
    res["multiturn"] = entry
    del layers, caches, ccalls
    torch.cuda.empty_cache()
    return res


def machine_info():
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "cpu_model": model,
            "affinity_cpus": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None}


def _oracle_threads():
    import threadpoolctl
    return max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] + [1])


def run_cpu_baselines(args, np, torch, configs, inputs, log, budget_s=2.0):
    """The fp64 oracle on the host cores for the other configurations, each on a bounded
    sample of one layer (one sequence of the batch, and for the 16384-token workload the
    first 2048 of its context tokens), repeated until budget_s is spent and scaled to the
    whole layer's keys (the oracle's work is linear in sequences x keys)."""
    import oracle as O

    out = {}

    def layer_sample(wl, T_full, B_full, T_sample, name, layer=0):
        gamma, w_q, w_k, w_v = (inputs.to_f64(t) for t in inputs.weights(wl, layer, 0, "cpu"))
        h, h_new = inputs.residuals(wl, layer, 1, T_sample, 0, "cpu")
        h, h_new = inputs.to_f64(h), inputs.to_f64(h_new)
        pos = np.arange(T_sample)[None, :]
        spent, n = 0.0, 0
        while spent < budget_s or n == 0:
            t0 = time.perf_counter()
            q, kt, vt = O.project_qkv(h_new, gamma, w_q, w_k, w_v, np.array([T_sample]), wl.n_q, wl.n_kv,
                                      wl.head_dim, wl.rms_eps, wl.rope_theta)
            O.kv_direct_decode(q, h, gamma, w_k, w_v, pos, kt[:, :, None], vt[:, :, None], wl.n_kv, wl.head_dim,
                               wl.rms_eps, wl.rope_theta)
            spent += time.perf_counter() - t0
            n += 1
        s_per = spent / n
        scale = (B_full * (T_full + 1)) / (T_sample + 1)
        layer_s = s_per * scale
        out[name] = {"workload": wl.name, "us_per_layer": layer_s * 1e6, "tok_s_per_layer": B_full / layer_s,
                     "sample": f"one sequence, {T_sample} context tokens + current, {n} runs in {spent:.2f} s; "
                               f"scaled x{scale:.1f} to B={B_full}, {T_full} + 1 keys"}
        log(f"[bench] cpu oracle {name}: {layer_s * 1e3:.1f} ms per layer")

    wl = configs.SMOLLM_FP32
    layer_sample(wl, wl.ctx, 1, wl.ctx, "smollm_fp32_layer")
    wl = configs.GEMMA3_SWEEP
    layer_sample(wl, wl.ctx, 1, wl.ctx, "gemma_ctx2048_b1_layer")
    out["gemma_ctx2048_b8_layer"] = dict(out["gemma_ctx2048_b1_layer"])
    for k in ("us_per_layer",):
        out["gemma_ctx2048_b8_layer"][k] *= 8
    out["gemma_ctx2048_b8_layer"]["tok_s_per_layer"] = out["gemma_ctx2048_b1_layer"]["tok_s_per_layer"]
    out["gemma_ctx2048_b8_layer"]["sample"] = "the B=1 sample above, scaled x8 (sequences are independent)"
    wl = configs.QWEN_1_5B
    layer_sample(wl, wl.ctx, wl.batch, 2048, "qwen_ctx16384_b8_layer")
    wl = configs.GEMMA3_MULTITURN
    for T in (256, 2560, 5120):
        layer_sample(wl, T, wl.batch, T, f"multiturn_b16_ctx{T}_layer")
    return {"kind": "oracle", "cores": _oracle_threads(), **machine_info(), "configs": out}


def run_cpu_baseline(args, np, wl, layers, T, B, inputs, log):
    """The fp64 oracle on the host cores: whole layers of the same decode step, taken
    in order and again from the first once all have run, until the time budget is
    spent; scaled to tokens/s of the full 34-layer step."""
    import threadpoolctl

    import oracle as O

    f = inputs.to_f64
    done, spent = 0, 0.0
    pos = np.arange(T)[None, :]
    for i in range(1 << 20):
        ly = layers[i % len(layers)]
        hx, hn = f(ly["h"]), f(ly["h_new"])
        g, wq, wk, wv = f(ly["gamma"]), f(ly["rw_q"]), f(ly["rw_k"]), f(ly["rw_v"])
        t0 = time.perf_counter()
        qo, kt, vt = O.project_qkv(hn, g, wq, wk, wv, np.array([T]), wl.n_q, wl.n_kv, wl.head_dim, wl.rms_eps,
                                   wl.rope_theta)
        O.kv_direct_decode(qo, hx, g, wk, wv, pos, kt[:, :, None], vt[:, :, None], wl.n_kv, wl.head_dim,
                           wl.rms_eps, wl.rope_theta)
        spent += time.perf_counter() - t0
        done += 1
        if spent >= args.cpu_seconds:
            break
    cores = max([i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()] + [1])
    log(f"[bench] cpu oracle: {done} layers in {spent:.1f} s on {cores} threads")
    return {"value": B * (done / wl.layers) / spent, "unit": "tok/s", "cores": cores, "kind": "oracle",
            **machine_info(),
            "sample": f"{done} layer evaluations ({done / wl.layers:.2f} steps of {wl.layers} layers) of the decode step (B={B}, {T} context tokens + current "
                      f"token), fp64 numpy oracle, scaled to the full step; {spent:.1f} s"}


if __name__ == "__main__":
    main()
