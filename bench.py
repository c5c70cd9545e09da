#!/usr/bin/env python3
"""Throughput of the DQT linear train step on one MI355X.

A step is the whole hot path over one batch: per-token activation
quantisation of each distinct layer input, the forward of every linear, both
backward products (dX and dW) of every linear, and the direct SR update of
every weight tensor -- all through the C ABI of libdqt on one HIP stream.

Default workload: the seven linears of a LLaMA block at hidden 768 / FFN 2048
(q, k, v, o 768x768; gate, up 768->2048; down 2048->768) over 8 x 1024 = 8192
tokens, ternary weights, bf16 activations and gradients, lr 3e-4.

Prints ONE JSON line.  `value` is step TFLOP/s (6 * M * d_in * d_out summed
over the linears, divided by the measured step time).  The step is captured
once as a HIP graph and replayed; per-kind durations (act-quant, forward, dX,
dW, SR) come from HIP events around back-to-back replays of a graph holding one
step's calls of that kind, on the same stream.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "i8": 5000.0, "fp8": 5000.0, "f32": 157.3}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="llama_h768")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--sr", choices=("fused", "separate"), default=None,
                   help="fused: the SR update consumes dW inside the backward call (dW is "
                        "never stored; bf16 environment only, the default there); separate: "
                        "backward writes dW, then the SR update call")
    p.add_argument("--cpu-tokens", type=int, default=8192,
                   help="tokens of the oracle's bounded sample")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="first run three plain device copies of MIB MiB, so that hardware "
                        "byte counters can be scaled against a kernel of known traffic")
    return p.parse_args()


class Block:
    """Device state of one workload: codes, inputs, outputs and scratch."""

    def __init__(self, wl, torch, dqt, W):
        self.wl = wl
        dev = "cuda:0"
        self.dev = dev
        bf = torch.bfloat16 if wl.x_dtype == "bf16" else torch.float32
        self.act = dqt.DQT_I8 if wl.act == "i8" else dqt.DQT_FP8E4M3
        self.xt = dqt.DQT_BF16 if wl.xt == "bf16" else dqt.DQT_F32
        wfmt = {"ternary": dqt.DQT_TERNARY2, "i4": dqt.DQT_INT4}.get(wl.wfmt, dqt.DQT_I8)
        M = wl.M
        self.weights, self.codes, self.dY, self.Y, self.dX, self.dW = [], [], [], [], [], []
        for li, lin in enumerate(wl.linears):
            W0, qdraw = W.weight_draws(wl, li)
            q, alpha = dqt.dqt_absmean_init(W0, wl.qmin, wl.qmax)
            if wl.init == "uniform":   # codes drawn directly; scale from W0 (qmax = 1)
                q = qdraw
            codes = (dqt.dqt_pack_ternary(q) if wl.wfmt == "ternary"
                     else dqt.dqt_pack_int4(q) if wl.wfmt == "i4" else q)
            self.codes.append(torch.from_numpy(np.ascontiguousarray(codes)).to(dev))
            self.weights.append(dqt.weight(lin.d_out, lin.d_in, wfmt, wl.qmin, wl.qmax, alpha, li))
            dy = torch.from_numpy(W.grad_draw(wl, li)).to(bf).to(dev)
            self.dY.append(dy)
            ydt = torch.bfloat16 if wl.y_out == "bf16" else torch.float32
            self.Y.append(torch.empty((M, lin.d_out), dtype=ydt, device=dev))
            dxdt = torch.bfloat16 if wl.dx_out == "bf16" else torch.float32
            self.dX.append(torch.empty((M, lin.d_in), dtype=dxdt, device=dev))
            self.dW.append(torch.empty((lin.d_out, lin.d_in), dtype=torch.float32, device=dev))
        self.X, self.Xq, self.xdq = {}, {}, {}
        qdt = torch.int8 if wl.act == "i8" else torch.uint8
        for name in wl.inputs:
            self.X[name] = torch.from_numpy(W.input_draw(wl, name)).to(bf).to(dev)
            self.Xq[name] = torch.empty((M, wl.input_width(name)), dtype=qdt, device=dev)
            self.xdq[name] = torch.empty((M,), dtype=torch.float32, device=dev)
        ents = []
        for li, lin in enumerate(wl.linears):
            ents.append(dict(w=self.weights[li], Wq=self.codes[li], Xq=self.Xq[lin.input],
                             xdq=self.xdq[lin.input], Y=self.Y[li], dY=self.dY[li],
                             dX=self.dX[li], dW=self.dW[li]))
        self.io_all = dqt.linear_io(ents)
        self.io_fused = dqt.linear_io([dict(e, dW=None) for e in ents])
        # AdamW moments (only the adamw_sr breakdown entry uses them)
        self.m = [torch.zeros_like(t) for t in self.dW]
        self.v = [torch.zeros_like(t) for t in self.dW]
        self.act_io = dqt.act_io([(self.X[n], self.Xq[n], self.xdq[n]) for n in wl.inputs])
        self.x_t = dqt.DQT_BF16 if wl.x_dtype == "bf16" else dqt.DQT_F32
        self.io_dx = dqt.linear_io([dict(e, dW=None) for e in ents])
        self.io_dw = dqt.linear_io([dict(e, dX=None) for e in ents])
        self.y_t = dqt.DQT_BF16 if wl.y_out == "bf16" else dqt.DQT_F32
        self.dy_t = dqt.DQT_BF16 if wl.dy_dtype == "bf16" else dqt.DQT_F32
        self.dx_t = dqt.DQT_BF16 if wl.dx_out == "bf16" else dqt.DQT_F32
        # one workspace serves every call: calls on one stream run in order
        ws = max(dqt.dqt_linear_bwd_batch_workspace(self.io_all, M),
                 dqt.dqt_linear_fwd_batch_workspace(self.io_all))
        self.ws = dqt.workspace(ws, dev)
        self.counters = torch.zeros((2,), dtype=torch.int64, device=dev)


def run_step(blk, dqt, step, stream, rec, split_bwd=False, sr="separate"):
    """Enqueue one train step: one batched call per stage (act-quant of every
    distinct input, forward, backward (dX and dW in one call, which may run
    them side by side), SR update) over all linears.  With sr == "fused" the
    backward and the SR update are one call (dW consumed where it is formed).
    With split_bwd the backward is two calls, dX then dW, so each can be
    timed on its own.  rec(kind, fn) runs fn (or records it into a graph)."""
    wl = blk.wl
    M = wl.M
    rec("act_quant", lambda: dqt.dqt_act_quant_batch(blk.act_io, blk.x_t, M, blk.act, stream))
    rec("fwd", lambda: dqt.dqt_linear_fwd_batch(blk.io_all, M, blk.act, blk.y_t, blk.ws, stream))
    if sr == "fused" and not split_bwd:
        rec("bwd_sr", lambda: dqt.dqt_linear_bwd_sr_batch(blk.io_fused, M, blk.act, blk.dy_t,
                                                          blk.xt, blk.dx_t, wl.lr, wl.seed, step,
                                                          blk.counters, blk.ws, stream))
        return
    if split_bwd:
        rec("bwd_dx", lambda: dqt.dqt_linear_bwd_batch(blk.io_dx, M, blk.act, blk.dy_t, blk.xt,
                                                       blk.dx_t, blk.ws, stream))
        rec("bwd_dw", lambda: dqt.dqt_linear_bwd_batch(blk.io_dw, M, blk.act, blk.dy_t, blk.xt,
                                                       blk.dx_t, blk.ws, stream))
    else:
        rec("bwd", lambda: dqt.dqt_linear_bwd_batch(blk.io_all, M, blk.act, blk.dy_t, blk.xt,
                                                    blk.dx_t, blk.ws, stream))
    rec("sr", lambda: dqt.dqt_sr_update_batch(blk.io_all, wl.lr, wl.seed, step, blk.counters,
                                              stream))


def algorithmic_units(wl):
    """Per step: flops of each GEMM stage, bytes of each streaming stage."""
    M = wl.M
    f = sum(2 * M * l.d_in * l.d_out for l in wl.linears)
    code_b = {"ternary": 0.25, "i4": 0.5}.get(wl.wfmt, 1.0)
    sr_bytes = sum((2 * code_b + 4) * l.d_in * l.d_out for l in wl.linears)
    # AdamW with SR: read g, m, v and the code; write m, v and the code
    adam_bytes = sum((2 * code_b + 20) * l.d_in * l.d_out for l in wl.linears)
    xb = 2 if wl.x_dtype == "bf16" else 4
    act_bytes = sum(M * wl.input_width(n) * (xb + 1) + 4 * M for n in wl.inputs)
    return {"fwd": f, "bwd": 2 * f, "bwd_sr": 2 * f, "bwd_dx": f, "bwd_dw": f, "sr": sr_bytes,
            "act_quant": act_bytes, "adamw_sr": adam_bytes, "upd_force": sr_bytes}


def cpu_baseline(wl, tokens: int, min_seconds: float = 10.0):
    """The oracle (untuned) on a bounded sample of the workload: one train step
    of every linear over the first `tokens` tokens, repeated until at least
    `min_seconds` of oracle time have accumulated (at most 5 repetitions)."""
    from threadpoolctl import threadpool_info

    from oracle import dqt_oracle as O
    from paper_2412_04787_amd import workloads as W

    tokens = min(tokens, wl.M)
    X = {n: W.input_draw(wl, n)[:tokens] for n in wl.inputs}
    prepared = []
    for li, lin in enumerate(wl.linears):
        W0, qdraw = W.weight_draws(wl, li)
        if wl.init == "uniform":
            q, alpha = qdraw, np.float32(O.absmean(W0))
        else:
            q, alpha = O.absmean_init(W0, wl.qmin, wl.qmax)
        dY = W.grad_draw(wl, li)[:tokens]
        x = X[lin.input]
        if wl.x_dtype == "bf16":
            x = O.bf16_to_f32(O.bf16_round(x))
            dY = O.bf16_to_f32(O.bf16_round(dY))
        prepared.append((li, lin, x, dY, q, alpha))
    flops = 0
    elapsed = 0.0
    reps = 0
    while reps < 5 and (reps == 0 or elapsed < min_seconds):
        for li, lin, x, dY, q, alpha in prepared:
            t0 = time.perf_counter()
            O.linear_train_step(x, dY, q, alpha, wl.qmin, wl.qmax, act=wl.act, xt=wl.xt,
                                y_out=wl.y_out, dx_out=wl.dx_out, lr=wl.lr, seed=wl.seed,
                                step=1, tensor_id=li)
            elapsed += time.perf_counter() - t0
            flops += 6 * tokens * lin.d_in * lin.d_out
        reps += 1
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    return {
        "value": flops / elapsed / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"{reps} x one train step (act-quant, fwd, dX, dW, SR) of all "
                  f"{len(wl.linears)} linears of {wl.name} over the first {tokens} of {wl.M} "
                  f"tokens; {elapsed:.1f} s of oracle time; host os.cpu_count()={os.cpu_count()}",
    }


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2412_04787_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def read_traffic(kernel_class: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel_class}_{workload}_counters.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            vals[k.strip()] = v.strip()
    if vals.get("kernel_source_hash") != kernel_source_hash():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1 "
                                   "(multi-GPU sharding is described, not built)"}))
        sys.exit(2)
    import torch

    from paper_2412_04787_amd import dqt, workloads as W

    dqt.load()
    wl = W.WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    if args.copy_calibration > 0:
        n = args.copy_calibration << 20
        src = torch.ones((n,), dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.sr is None:
        args.sr = "fused" if wl.xt == "bf16" and wl.dy_dtype == "bf16" else "separate"
    blk = Block(wl, torch, dqt, W)
    units = algorithmic_units(wl)

    def plain(kind, fn):
        fn()

    for s in range(args.warmup):
        run_step(blk, dqt, 1000 + s, None, plain, sr=args.sr)
    torch.cuda.synchronize()

    # One step is ~40 kernel launches; on its own the host would need longer
    # to issue them than the GPU needs to run them, so the step is captured
    # once into a HIP graph and the timed region replays it.  Every kernel of
    # the step runs in every replay.
    step_graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(step_graph):
        run_step(blk, dqt, 1, None, plain, sr=args.sr)
    torch.cuda.synchronize()
    step_graph.replay()
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    start.record(stream)
    for _ in range(args.steps):
        step_graph.replay()
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps

    # Per-call-kind durations: a graph holding one step's calls of one kind,
    # replayed back to back between two events on the same stream.  The
    # step's own calls first; then dX and dW each in a call of its own.
    step_kinds = ["act_quant", "fwd"] + (["bwd_sr"] if args.sr == "fused" else ["bwd", "sr"])
    kinds = step_kinds + (["bwd", "sr"] if args.sr == "fused" else []) + ["bwd_dx", "bwd_dw",
                                                                         "adamw_sr", "upd_force"]
    var_ws = dqt.workspace(dqt.dqt_update_variant_workspace(len(wl.linears)))
    adam_hp = dqt.adamw(wl.lr, 0.9, 0.95, 1e-8, 0.1)
    per_kind_ms, per_kind_units, per_kind_n = {}, {}, {}
    for kind in kinds:
        calls = []

        def only(k, fn, kind=kind, calls=calls):
            if k == kind:
                calls.append(k)
                fn()

        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            if kind == "upd_force":
                # force-to-update of the smallest 20 % (exact selection, then the update)
                calls.append(kind)
                dqt.dqt_update_variant_batch(blk.io_all, wl.lr, wl.seed, 1, dqt.DQT_UPD_FORCE_CHANGE,
                                             0.2, blk.counters, var_ws)
            elif kind == "adamw_sr":
                # the AdamW variant of the update (not part of the step)
                calls.append(kind)
                dqt.dqt_adamw_sr_update_batch(blk.io_all, blk.m, blk.v, adam_hp, wl.seed, 1,
                                              blk.counters, None)
            else:
                run_step(blk, dqt, 1, None, only, split_bwd=kind in ("bwd_dx", "bwd_dw"),
                         sr="fused" if kind == "bwd_sr" else "separate")
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        per_kind_ms[kind] = e0.elapsed_time(e1)
        per_kind_units[kind] = args.steps * units[kind]
        per_kind_n[kind] = args.steps * len(calls)
        del g

    flops = wl.train_flops
    value = flops / (ms_per_step * 1e-3) / 1e12
    gemm_dtype = {"fwd": "fp8" if wl.act == "e4m3" else "i8",
                  "bwd": "bf16" if wl.dy_dtype == "bf16" and wl.xt == "bf16" else "f32",
                  "bwd_sr": "bf16",
                  "bwd_dx": "bf16" if wl.dy_dtype == "bf16" else "f32",
                  "bwd_dw": "bf16" if wl.xt == "bf16" else "f32"}
    breakdown = {}
    for kind in per_kind_ms:
        t = per_kind_ms[kind] / args.steps
        u = per_kind_units[kind] / args.steps
        entry = {"ms_per_step": round(t, 4), "calls_per_step": per_kind_n[kind] // args.steps}
        if kind in gemm_dtype:
            tf = u / (t * 1e-3) / 1e12
            entry.update({"tflops": round(tf, 1), "dtype": gemm_dtype[kind],
                          "frac_peak": round(tf / PEAK_TFLOPS[gemm_dtype[kind]], 4)})
        else:
            gbs = u / (t * 1e-3) / 1e9
            entry.update({"gbs": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)})
        breakdown[kind] = entry

    # the dominant kernel class: largest share of the step
    dom = max(step_kinds, key=lambda k: per_kind_ms[k])
    dom_avg_ms = per_kind_ms[dom] / per_kind_n[dom]
    dom_units = per_kind_units[dom] / per_kind_n[dom]
    if dom in gemm_dtype:
        achieved = dom_units / (dom_avg_ms * 1e-3) / 1e12
        peak = PEAK_TFLOPS[gemm_dtype[dom]]
        roof = {"bound": "mfma", "unit": "TFLOP/s"}
    else:
        achieved = dom_units / (dom_avg_ms * 1e-3) / 1e9
        peak = PEAK_HBM_GBS
        roof = {"bound": "hbm", "unit": "GB/s"}
    traffic = read_traffic(dom, wl.name)
    roof.update({"kernel": dom, "achieved": round(achieved, 2), "peak": peak,
                 "frac": round(achieved / peak, 4), "traffic": traffic,
                 "avg_launch_ms": round(dom_avg_ms, 5), "units_per_launch": dom_units})

    sr_t = per_kind_ms.get("sr", 0.0) / args.steps
    sr_gbs = per_kind_units.get("sr", 0.0) / args.steps / (sr_t * 1e-3) / 1e9 if sr_t else None
    mfma_frac = sum(per_kind_units[k] / args.steps / (PEAK_TFLOPS[gemm_dtype[k]] * 1e12)
                    for k in ("fwd", "bwd_dx", "bwd_dw")) / (ms_per_step * 1e-3)

    out = {
        "metric": "DQT linear train-step TFLOP/s (fwd+bwd) + SR-update GB/s, % of MI355X peak",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8+bf16" if wl.act == "i8" and wl.xt == "bf16" else f"{wl.act}+{wl.xt}",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: LLaMA-block linears q,k,v,o {wl.linears[0].d_in}x"
                        f"{wl.linears[0].d_out}, gate/up {wl.linears[4].d_in}->"
                        f"{wl.linears[4].d_out}, down {wl.linears[6].d_in}->"
                        f"{wl.linears[6].d_out}; {wl.M} tokens; {wl.wfmt} weights; "
                        f"{wl.act} activations; {wl.xt} environment; lr {wl.lr}",
            "tokens": wl.M, "linears": len(wl.linears), "weights": wl.n_weights,
            "sr_update": "fused into the dW product" if args.sr == "fused" else "separate call",
            "parallelism": "single GPU",
        },
        "sr_update_gbs": round(sr_gbs, 1) if sr_gbs else None,
        "sr_update_frac_hbm": round(sr_gbs / PEAK_HBM_GBS, 4) if sr_gbs else None,
        "gemm_frac_of_dtype_peak": round(mfma_frac, 4),
        "breakdown": breakdown,
        "wall_s_timed_region": round(wall, 3),
        "roofline": roof,
        "kernel_source_hash": kernel_source_hash(),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_tokens)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
