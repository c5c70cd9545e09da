#!/usr/bin/env python3
"""Throughput of the DQT linear train step on one MI355X.

A step is the whole hot path over one batch: per-token activation
quantisation of each distinct layer input, the forward of every linear, both
backward products (dX and dW) of every linear, and the direct SR update of
every weight tensor -- all through the C ABI of libdqt on one HIP stream.

Default workload: the seven linears of a LLaMA block at hidden 4096 / FFN
11008 (q, k, v, o 4096x4096; gate, up 4096->11008; down 11008->4096) over
8192 tokens, ternary weights, e4m3 activations, bf16 environment, lr 1e-4:
the largest of the single-block workloads.

Prints ONE JSON line.  `value` is step TFLOP/s (6 * M * d_in * d_out summed
over the linears, divided by the measured step time).  The step is captured
once as a HIP graph; K replays are timed between two events (ms_per_step),
with an event after every replay for the median and p10 / p90.  Per-kind
durations (act-quant, forward, the backward calls, the SR update) come from
HIP events around replays of a graph holding one step's calls of that kind,
on the same stream; the SR update call rotates over enough copies of codes
and gradients (more than 512 MB in all) that the 256 MB last-level cache
cannot serve one call's data to the next.
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
# bytes of code storage per weight
CODE_BYTES = {"ternary": 0.25, "i3": 0.375, "i4": 0.5, "i8": 1.0}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="llama_h4096")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--sr", choices=("fused", "separate"), default=None,
                   help="fused: the SR update consumes dW inside the backward call (dW is "
                        "never stored; bf16 environment only, the default there); separate: "
                        "backward writes dW, then the SR update call")
    p.add_argument("--cpu-tokens", type=int, default=256,
                   help="tokens of the oracle's GEMM slab (all cores); a slab of a quarter of "
                        "that many tokens is timed on one thread")
    p.add_argument("--cpu-sr-weights", type=int, default=16 << 20,
                   help="weights of the oracle's SR sample")
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
        wfmt = {"ternary": dqt.DQT_TERNARY2, "i4": dqt.DQT_INT4, "i3": dqt.DQT_INT3}.get(wl.wfmt,
                                                                                   dqt.DQT_I8)
        M = wl.M
        self.weights, self.codes, self.dY, self.Y, self.dX, self.dW = [], [], [], [], [], []
        for li, lin in enumerate(wl.linears):
            W0, qdraw = W.weight_draws(wl, li)
            q, alpha = dqt.dqt_absmean_init(W0, wl.qmin, wl.qmax)
            if wl.init == "uniform":   # codes drawn directly; scale from W0 (qmax = 1)
                q = qdraw
            codes = (dqt.dqt_pack_ternary(q) if wl.wfmt == "ternary"
                     else dqt.dqt_pack_int4(q) if wl.wfmt == "i4"
                     else dqt.dqt_pack_int3(q) if wl.wfmt == "i3" else q)
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


def gemm_min_bytes(wl):
    """Per GEMM call kind, the bytes it moves at the least: each operand read
    once and each output written once (quantised inputs once per distinct
    input; the fused call reads and writes the codes instead of writing dW)."""
    M = wl.M
    cb = CODE_BYTES.get(wl.wfmt, 1.0)
    size = {"f32": 4, "bf16": 2}
    xq = sum(M * wl.input_width(n) for n in wl.inputs) + 4 * M * len(wl.inputs)
    y = sum(M * l.d_out * size[wl.y_out] for l in wl.linears)
    dy = sum(M * l.d_out * size[wl.dy_dtype] for l in wl.linears)
    dx = sum(M * l.d_in * size[wl.dx_out] for l in wl.linears)
    codes = cb * wl.n_weights
    dw = 4 * wl.n_weights
    return {"fwd": xq + codes + y, "bwd_dx": dy + codes + dx, "bwd_dw": dy + xq + dw,
            "bwd": dy + xq + codes + dx + dw, "bwd_sr": dy + xq + 2 * codes + dx}


def algorithmic_units(wl):
    """Per step: flops of each GEMM stage, bytes of each streaming stage."""
    M = wl.M
    f = sum(2 * M * l.d_in * l.d_out for l in wl.linears)
    code_b = CODE_BYTES.get(wl.wfmt, 1.0)
    sr_bytes = sum((2 * code_b + 4) * l.d_in * l.d_out for l in wl.linears)
    # AdamW with SR: read g, m, v and the code; write m, v and the code
    adam_bytes = sum((2 * code_b + 20) * l.d_in * l.d_out for l in wl.linears)
    xb = 2 if wl.x_dtype == "bf16" else 4
    act_bytes = sum(M * wl.input_width(n) * (xb + 1) + 4 * M for n in wl.inputs)
    # force-to-update of the smallest 20 %: three selection passes over the
    # gradient (4 B per weight each), then the update
    upd_bytes = sr_bytes + 3 * 4 * wl.n_weights
    return {"fwd": f, "bwd": 2 * f, "bwd_sr": 2 * f, "bwd_dx": f, "bwd_dw": f, "sr": sr_bytes,
            "act_quant": act_bytes, "adamw_sr": adam_bytes, "upd_force": upd_bytes}


def _oracle_slab(O, W, wl, tokens):
    """The oracle's inputs for one slab of `tokens` tokens: per linear (lin,
    x, dY, q, alpha) with the environment's bf16 rounding applied."""
    # (the first `tokens` rows of each draw: the generator fills rows in order)
    X = {n: W.input_draw(wl, n, M=tokens) for n in wl.inputs}
    prepared = []
    for li, lin in enumerate(wl.linears):
        W0, qdraw = W.weight_draws(wl, li)
        if wl.init == "uniform":
            q, alpha = qdraw, np.float32(O.absmean(W0))
        else:
            q, alpha = O.absmean_init(W0, wl.qmin, wl.qmax)
        dY = W.grad_draw(wl, li, M=tokens)
        x = X[lin.input]
        if wl.x_dtype == "bf16":
            x = O.bf16_to_f32(O.bf16_round(x))
            dY = O.bf16_to_f32(O.bf16_round(dY))
        prepared.append((li, lin, x, dY, q, alpha))
    return prepared


def _time_oracle_gemms(O, wl, prepared):
    """Seconds for act-quant, forward, dX and dW of every linear of a slab."""
    t = 0.0
    for li, lin, x, dY, q, alpha in prepared:
        t0 = time.perf_counter()
        Xq, d = O.act_quant(x, wl.act)
        O.linear_fwd(Xq, d, wl.act, q, alpha, wl.y_out)
        O.linear_bwd(dY, q, alpha, Xq, d, wl.act, wl.xt, wl.dx_out)
        t += time.perf_counter() - t0
    return t


def cpu_baseline(wl, tokens: int, sr_weights: int):
    """The oracle (untuned) timed on the host cores on a bounded sample of
    the workload, extrapolated to one whole step:
      * the GEMM part (act-quant, forward, dX, dW of every linear) on a slab
        of the first `tokens` tokens with every BLAS thread, and on a slab of
        tokens // 4 tokens on one thread; each scaled by M / slab tokens;
      * the SR update on `sr_weights` weights (the same share of every
        tensor, on its real gradient-sized draws), scaled by all weights /
        sampled weights.
    value = the step's flops / (GEMM time + SR time), all cores."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import dqt_oracle as O
    from paper_2412_04787_amd import workloads as W

    tokens = max(16, min(tokens, wl.M))
    tok1 = max(16, tokens // 4)
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    prepared = _oracle_slab(O, W, wl, tokens)
    t_all = _time_oracle_gemms(O, wl, prepared)
    small = [(li, lin, x[:tok1], dY[:tok1], q, a) for li, lin, x, dY, q, a in prepared]
    with threadpool_limits(limits=1):
        t_one = _time_oracle_gemms(O, wl, small)
    # SR sample: the first rows of every tensor, in proportion to its size
    share = min(1.0, sr_weights / wl.n_weights)
    rng = np.random.default_rng(0)
    t_sr, sampled = 0.0, 0
    for li, lin, x, dY, q, alpha in prepared:
        rows = max(1, int(round(share * lin.d_out)))
        qs = np.ascontiguousarray(q[:rows])
        g = (rng.standard_normal(qs.shape, dtype=np.float32) * np.float32(1e-2 * tokens ** 0.5))
        t0 = time.perf_counter()
        O.sr_update(qs.ravel(), g.ravel(), wl.lr, alpha, wl.qmin, wl.qmax, wl.seed, 1, li)
        t_sr += time.perf_counter() - t0
        sampled += qs.size
    sr_full = t_sr * wl.n_weights / sampled
    gemm_all = t_all * wl.M / tokens
    gemm_one = t_one * wl.M / tok1
    flops = wl.train_flops
    return {
        "value": flops / (gemm_all + sr_full) / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"extrapolated: act-quant/fwd/dX/dW of all {len(wl.linears)} linears of "
                   f"{wl.name} on the first {tokens} of {wl.M} tokens ({t_all:.1f} s on {threads} "
                   f"BLAS threads, x {wl.M / tokens:g}) plus the SR update on {sampled} of "
                   f"{wl.n_weights} weights ({t_sr:.1f} s on one thread, x "
                   f"{wl.n_weights / sampled:.1f}); host os.cpu_count()={os.cpu_count()}"),
        "step_s_all_cores": round(gemm_all + sr_full, 2),
        "step_s_one_thread": round(gemm_one + sr_full, 2),
        "one_thread_value": flops / (gemm_one + sr_full) / 1e12,
        "one_thread_sample": f"GEMM part on the first {tok1} tokens ({t_one:.1f} s, x {wl.M / tok1:g})",
        "sr_update_gbs_one_thread": round(
            sum((2 * CODE_BYTES.get(wl.wfmt, 1.0) + 4) * l.d_in * l.d_out
                for l in wl.linears) / sr_full / 1e9, 3),
    }


def kernel_source_hash() -> str:
    """Hash of what the kernels are built from: the HIP sources and the build
    script (its compiler flags)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2412_04787_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            h.update(open(os.path.join(csrc, f), "rb").read())
    h.update(open(os.path.join(ROOT, "paper_2412_04787_amd", "build_lib.py"), "rb").read())
    return h.hexdigest()[:16]


def read_traffic(kernel_class: str, workload: str, kernel_only: bool = False):
    """Bytes per launch that the L2 caches fetched from and wrote to memory
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of known size), from the
    committed rocprofv3 counter summary, if it was taken on the current
    kernel sources; else None.  kernel_only: the GEMM kernel's own bytes,
    without the passes of its call.  The counters see the last-level cache
    (MALL) and HBM alike, so on a block whose data fits the 256 MB MALL this
    is an upper bound of the HBM bytes."""
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
        return float(vals["gemm_kernel_fetch_write_bytes" if kernel_only else "fetch_write_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def model_cpu_baseline(cfg, tokens: int, sr_weights: int):
    """The oracle on one block's seven DQT linears (the model's shapes, its
    ternary codes and lr), extrapolated by the model's layer count.  The
    attention, norms, embedding and LM head are not DQT linears and have no
    oracle; the value is the DQT part's flops over that time."""
    import dataclasses

    from paper_2412_04787_amd import workloads as W
    lin = []
    for _, grp in cfg.linears():
        for name, d_in, d_out in grp:
            lin.append(W.Linear(name, d_in, d_out, "mlp_hidden" if name == "down" else
                                "attn_out" if name == "o" else
                                "attn_in" if name in ("q", "k", "v") else "mlp_in"))
    wl = dataclasses.replace(W.WORKLOADS["llama_h2048"], name=f"{cfg.name} block", M=cfg.tokens,
                             linears=tuple(lin), wfmt="ternary", qmin=-1, qmax=1, lr=cfg.lr)
    b = cpu_baseline(wl, tokens, max(1, sr_weights))
    L = cfg.layers
    # every layer has the block's flops and its time: the rate is the block's
    b["step_s_all_cores"] = round(b["step_s_all_cores"] * L, 2)
    b["step_s_one_thread"] = round(b["step_s_one_thread"] * L, 2)
    b["sample"] = (f"per-layer extrapolation x {L} of one block's DQT linears (the model's "
                   f"attention, norms, embedding and LM head are not DQT linears and are not "
                   f"in the oracle); block: " + b["sample"])
    return b


def run_model(args):
    """A train step of the whole model (model_step.py): forward, backward
    with the SR update of every DQT tensor, AdamW on the dense parameters."""
    import torch

    from paper_2412_04787_amd import dqt, model_step as MS

    cfg = MS.MODELS[args.workload]
    torch.cuda.set_device(0)
    model = MS.DQTModel(cfg)
    flops = cfg.step_flops()
    losses = []
    for s in range(args.warmup):
        tok, tgt = MS.synthetic_batch(cfg, s)
        losses.append(float(model.train_step(tok, tgt).item()))
        print(f"warmup step {s + 1}: loss {losses[-1]:.4f}", file=sys.stderr, flush=True)
    batches = [MS.synthetic_batch(cfg, args.warmup + s) for s in range(args.steps)]
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    changed = []
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev[0].record(stream)
    step_losses = []
    c0 = model.counters.clone()
    for s in range(args.steps):
        step_losses.append(model.train_step(*batches[s]))
        ev[s + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    per = [ev[s].elapsed_time(ev[s + 1]) for s in range(args.steps)]
    total_ms = ev[0].elapsed_time(ev[args.steps])
    losses += [float(x.item()) for x in step_losses]
    changed = int((model.counters - c0)[0].item())
    ms = total_ms / args.steps
    pct = lambda v, q: float(np.percentile(np.asarray(v), q))
    value = flops["total"] / (ms * 1e-3) / 1e12
    out = {
        "metric": "DQT model train-step TFLOP/s (fwd+bwd of the whole model, SR update of every "
                  "DQT weight in the step)",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "ms_per_step_median": round(pct(per, 50), 3),
        "ms_per_step_p10": round(pct(per, 10), 3),
        "ms_per_step_p90": round(pct(per, 90), 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8+bf16",
        "data": "synthetic (uniform-random token ids)",
        "config": {
            "workload": f"{cfg.name}: {cfg.layers}-layer LLaMA-shaped model, hidden {cfg.hidden}, "
                        f"{cfg.heads} heads, FFN {cfg.ffn}, vocab {cfg.vocab}, RMSNorm, RoPE; "
                        f"all {7 * cfg.layers} block linears DQT ternary (int8 activations, "
                        f"bf16 environment); batch {cfg.batch} x seq {cfg.seq}; lr {cfg.lr}",
            "tokens": cfg.tokens, "dqt_weights": cfg.dqt_weights,
            "sr_update": "fused into each layer's dW product (one backward call per group of "
                         "linears sharing an input)",
            "parallelism": "single GPU",
        },
        "flops_per_step": flops,
        "dqt_tflops_share": round(flops["dqt_linears"] / (ms * 1e-3) / 1e12, 2),
        "losses": [round(x, 4) for x in losses],
        "loss_expected_at_init": round(MS.initial_loss_expected(cfg), 4),
        "weights_changed_per_step": changed / args.steps,
        "update_fraction_per_step": round(changed / args.steps / cfg.dqt_weights, 6),
        "wall_s_timed_region": round(wall, 3),
        "kernel_source_hash": kernel_source_hash(),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = model_cpu_baseline(cfg, args.cpu_tokens, args.cpu_sr_weights // 4)
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this library runs on one GPU only; --gpus must be 1 "
                                   "(multi-GPU sharding is described, not built)"}))
        sys.exit(2)
    from paper_2412_04787_amd import model_step

    if args.workload in model_step.MODELS:
        run_model(args)
        return
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

    def time_graph(g, reps):
        """Replays g `reps` times on `stream`: (total ms, per-replay ms list)."""
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for r in range(reps):
            g.replay()
            ev[r + 1].record(stream)
        torch.cuda.synchronize()
        per = [ev[r].elapsed_time(ev[r + 1]) for r in range(reps)]
        return ev[0].elapsed_time(ev[reps]), per

    # the timed region: exactly K replays of the whole step
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    total_ms, per_step = time_graph(step_graph, args.steps)
    wall = time.perf_counter() - wall0
    ms_per_step = total_ms / args.steps
    pct = lambda v, q: float(np.percentile(np.asarray(v), q))

    # Per-call-kind durations: a graph holding one step's calls of one kind,
    # replayed between events on the same stream.  The step's own calls
    # first; then dX and dW each in a call of its own, the SR update call
    # (over rotating buffer sets), AdamW with SR and an analysis variant.
    step_kinds = ["act_quant", "fwd"] + (["bwd_sr"] if args.sr == "fused" else ["bwd", "sr"])
    kinds = step_kinds + (["bwd", "sr"] if args.sr == "fused" else []) + ["bwd_dx", "bwd_dw",
                                                                         "adamw_sr", "upd_force"]
    var_ws = dqt.workspace(dqt.dqt_update_variant_workspace(len(wl.linears)))
    adam_hp = dqt.adamw(wl.lr, 0.9, 0.95, 1e-8, 0.1)
    # SR rotation: copies of the codes and of the gradient (the backward's dW,
    # filled by the "bwd" kind, which runs before "sr") until more than
    # 512 MB are in the rotation
    set_bytes = units["sr"]
    n_sets = max(2, int(np.ceil(600e6 / set_bytes)))
    sr_sets = []
    per_kind = {}
    for kind in kinds:
        calls = []

        def only(k, fn, kind=kind, calls=calls):
            if k == kind:
                calls.append(k)
                fn()

        if kind == "sr" and not sr_sets:
            torch.cuda.synchronize()
            for si in range(n_sets):
                if si == 0:
                    sr_sets.append(blk.io_all)
                    continue
                ents = []
                for li in range(len(wl.linears)):
                    ents.append(dict(w=blk.weights[li], Wq=blk.codes[li].clone(),
                                     dW=blk.dW[li].clone()))
                sr_sets.append(dqt.linear_io(ents))
            torch.cuda.synchronize()
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
            elif kind == "sr":
                for io in sr_sets:
                    calls.append(kind)
                    dqt.dqt_sr_update_batch(io, wl.lr, wl.seed, 1, blk.counters)
            else:
                run_step(blk, dqt, 1, None, only, split_bwd=kind in ("bwd_dx", "bwd_dw"),
                         sr="fused" if kind == "bwd_sr" else "separate")
        torch.cuda.synchronize()
        g.replay()                      # one untimed replay
        tot, per = time_graph(g, args.steps)
        n_calls = len(calls)
        per_kind[kind] = {"mean": tot / args.steps / n_calls, "calls": n_calls,
                          "median": pct(per, 50) / n_calls, "p10": pct(per, 10) / n_calls,
                          "p90": pct(per, 90) / n_calls}
        del g

    flops = wl.train_flops
    value = flops / (ms_per_step * 1e-3) / 1e12
    gemm_dtype = {"fwd": "fp8" if wl.act == "e4m3" else "i8",
                  "bwd": "bf16" if wl.dy_dtype == "bf16" and wl.xt == "bf16" else "f32",
                  "bwd_sr": "bf16",
                  "bwd_dx": "bf16" if wl.dy_dtype == "bf16" else "f32",
                  "bwd_dw": "bf16" if wl.xt == "bf16" else "f32"}
    breakdown = {}
    min_bytes = gemm_min_bytes(wl)
    for kind, tk in per_kind.items():
        t = tk["median"]
        u = units[kind]
        entry = {"ms_per_call": round(t, 4), "p10_ms": round(tk["p10"], 4),
                 "p90_ms": round(tk["p90"], 4), "calls_per_step": 1}
        if kind == "sr":
            entry["buffer_sets_rotated"] = tk["calls"]
        if kind in gemm_dtype:
            tf = u / (t * 1e-3) / 1e12
            # the call's roofline bound: max(flops at the dtype's peak, least
            # bytes at 8 TB/s)
            bound_ms = max(u / (PEAK_TFLOPS[gemm_dtype[kind]] * 1e12),
                           min_bytes[kind] / (PEAK_HBM_GBS * 1e9)) * 1e3
            entry.update({"tflops": round(tf, 1), "dtype": gemm_dtype[kind],
                          "frac_peak": round(tf / PEAK_TFLOPS[gemm_dtype[kind]], 4),
                          "bound_ms": round(bound_ms, 4), "frac_of_bound": round(bound_ms / t, 4)})
        else:
            gbs = u / (t * 1e-3) / 1e9
            entry.update({"gbs": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)})
        breakdown[kind] = entry

    # the dominant call of the step: its share of the step is the largest.
    # A GEMM call is its GEMM kernel launch plus passes around it (operand
    # expansion or transposition, the tile-counter clear); the roofline is the
    # GEMM kernel's own: the library's launch timer brackets each GEMM kernel
    # launch with HIP events on the call's stream, here over `steps` calls of
    # the dominant kind issued back to back.
    dom = max(step_kinds, key=lambda k: per_kind[k]["median"])
    dom_call_ms = per_kind[dom]["mean"]
    dom_units = units[dom]
    kernel_ms, launches = None, 0
    if dom in gemm_dtype:
        def only_dom(k, fn):
            if k == dom:
                fn()
        cap = 8 * args.steps
        torch.cuda.synchronize()
        dqt.dqt_launch_timer_start(cap)
        try:
            for r in range(args.steps):
                run_step(blk, dqt, 3000 + r, None, only_dom, split_bwd=dom in ("bwd_dx", "bwd_dw"),
                         sr="fused" if dom == "bwd_sr" else "separate")
            torch.cuda.synchronize()
        finally:
            launch_ms, launches = dqt.dqt_launch_timer_stop(cap)
        if launches > 0 and launches % args.steps == 0:
            kernel_ms = sum(launch_ms) / args.steps
    dom_avg_ms = kernel_ms if kernel_ms is not None else dom_call_ms
    if dom in gemm_dtype:
        achieved = dom_units / (dom_avg_ms * 1e-3) / 1e12
        peak = PEAK_TFLOPS[gemm_dtype[dom]]
        roof = {"bound": "mfma", "unit": "TFLOP/s"}
    else:
        achieved = dom_units / (dom_avg_ms * 1e-3) / 1e9
        peak = PEAK_HBM_GBS
        roof = {"bound": "hbm", "unit": "GB/s"}
    traffic = read_traffic(dom, wl.name, kernel_only=kernel_ms is not None)
    roof.update({"achieved": round(achieved, 2), "peak": peak,
                 "frac": round(achieved / peak, 4), "traffic": traffic, "kernel": dom,
                 "avg_launch_ms": round(dom_avg_ms, 5), "units_per_launch": dom_units,
                 "timing": ("GEMM kernel launches (library launch timer)" if kernel_ms is not None
                            else "whole call"),
                 "gemm_launches_per_call": launches // args.steps if kernel_ms is not None else None,
                 "call_ms": round(dom_call_ms, 5)})

    # The chip's own streaming read rate (a plain one-pass read, 16-byte
    # non-temporal loads, alternating two 1 GiB buffers): what the SR update,
    # a stream of 4.25 B read and 0.25 B written per ternary weight, can
    # approach at best.
    rs_bytes = 1 << 30
    rs_bufs = [torch.full((rs_bytes // 4,), r + 1, dtype=torch.int32, device="cuda:0") for r in range(2)]
    rs_sink = torch.empty((dqt.READ_STREAM_SINK_WORDS,), dtype=torch.int32, device="cuda:0")
    for r in range(4):
        dqt.dqt_read_stream(rs_bufs[r & 1], rs_sink)
    rs_ev = [torch.cuda.Event(enable_timing=True) for _ in range(21)]
    torch.cuda.synchronize()
    rs_ev[0].record(stream)
    for r in range(20):
        dqt.dqt_read_stream(rs_bufs[r & 1], rs_sink, stream)
        rs_ev[r + 1].record(stream)
    torch.cuda.synchronize()
    read_gbs = rs_bytes / (pct([rs_ev[r].elapsed_time(rs_ev[r + 1]) for r in range(20)], 50) * 1e-3) / 1e9
    del rs_bufs, rs_sink

    sr = breakdown.get("sr")
    mfma_frac = sum(units[k] / (PEAK_TFLOPS[gemm_dtype[k]] * 1e12)
                    for k in ("fwd", "bwd_dx", "bwd_dw")) / (ms_per_step * 1e-3)

    out = {
        "metric": "DQT linear train-step TFLOP/s (fwd+bwd) + SR-update GB/s, % of MI355X peak",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_median": round(pct(per_step, 50), 4),
        "ms_per_step_p10": round(pct(per_step, 10), 4),
        "ms_per_step_p90": round(pct(per_step, 90), 4),
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
        "sr_update_gbs": sr["gbs"] if sr else None,
        "sr_update_frac_hbm": sr["frac_hbm"] if sr else None,
        "sr_update_note": (f"separate SR call, median over {args.steps} replays, rotating "
                           f"{n_sets} buffer sets of {set_bytes / 1e6:.1f} MB") if sr else None,
        "hbm_read_stream_gbs": round(read_gbs, 1),
        "hbm_read_stream_frac_hbm": round(read_gbs / PEAK_HBM_GBS, 4),
        "sr_update_frac_of_read_stream": round(sr["gbs"] / read_gbs, 4) if sr else None,
        "gemm_frac_of_dtype_peak": round(mfma_frac, 4),
        "breakdown": breakdown,
        "wall_s_timed_region": round(wall, 3),
        "roofline": roof,
        "kernel_source_hash": kernel_source_hash(),
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_tokens, args.cpu_sr_weights)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
