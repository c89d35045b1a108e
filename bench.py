"""Benchmark: Dyad feed-forward fwd+bwd on one MI355X.

One step = for each of Dyad-IT, -OT, -DT, the feed-forward block of the chosen
workload (default: OPT-125m shapes, fc1 768->3072 with GELU, fc2 3072->768,
n_dyad=4, M=16384 tokens, bf16 with fp32 accumulation) run forward and
backward through libdyad: fc1 fwd (GELU, pre-activation stashed), fc2 fwd,
fc2 dX (GELU' fused), fc2 dW+db, fc1 dX, fc1 dW+db.  FLOPs are counted
algorithmically, 4*M*n_in*n_out/n_dyad per pass.

Prints one JSON line.  Inputs are seeded synthetic tensors already resident
in HBM when the timed region starts.
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

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="opt125m_ff")
    ap.add_argument("--variants", default="IT,OT,DT")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=2048)
    return ap.parse_args()


def workload(name):
    import workloads as W
    table = {w.name: w for w in [W.OPT125M, W.OPT350M, W.TINY, *W.SWEEP, *W.WIDE]}
    if name not in table:
        raise SystemExit(f"unknown workload {name}; choose from {sorted(table)}")
    return table[name]


class Layer:
    """Device buffers of one Dyad layer, allocated once."""

    def __init__(self, dy, torch, n_in, n_out, D, M, act, seed_offset, dev):
        from workloads import layer_inputs
        L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=seed_offset)
        self.n_in, self.n_out, self.D, self.M, self.act = n_in, n_out, D, M, act
        self.W1, self.W2, self.b = L.W1.to(dev), L.W2.to(dev), L.bias.to(dev)
        self.dW1, self.dW2 = torch.empty_like(self.W1), torch.empty_like(self.W2)
        self.db = torch.empty_like(self.b)
        self.X0 = L.X.to(dev)      # input of the first layer
        self.dZ0 = L.dZ.to(dev)    # upstream gradient of the last layer
        self.Y = torch.empty((M, n_out), dtype=torch.bfloat16, device=dev)
        self.H = torch.empty_like(self.Y) if act else None
        self.dX = torch.empty((M, n_in), dtype=torch.bfloat16, device=dev)
        self.flops = 4.0 * M * n_in * n_out / D


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    import paper_2312_06881_amd as dy

    wl = workload(args.workload)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lib = dy._load()
    stream = torch.cuda.current_stream(dev)
    sp = stream.cuda_stream
    D, M = wl.n_dyad, wl.M
    variants = [v for v in args.variants.split(",") if v]
    vid = {"IT": dy.IT, "OT": dy.OT, "DT": dy.DT}

    (n1, i1, o1), (n2, i2, o2) = wl.layers if len(wl.layers) == 2 else (wl.layers[0], wl.layers[0])
    fc1 = Layer(dy, torch, i1, o1, D, M, True, 0, dev)
    fc2 = Layer(dy, torch, i2, o2, D, M, False, 1, dev)
    ws_bytes = max(dy.dyad_dw_workspace_bytes(vid[v], L.n_in, L.n_out, D, M, dy.BF16)
                   for v in variants for L in (fc1, fc2))
    ws = torch.empty((max(ws_bytes, 16),), dtype=torch.uint8, device=dev)

    def p(t):
        return None if t is None else t.data_ptr()

    def check(rc):
        if rc != 0:
            raise RuntimeError(dy.dyad_strerror(rc))

    # one call = one entry point of the C-ABI; kind: "gemm" (fwd / dX) or "dw"
    def calls(v):
        V = vid[v]
        return [
            ("gemm", fc1.flops, lambda: lib.dyad_forward(V, fc1.n_in, fc1.n_out, D, M, dy.BF16,
                                                        p(fc1.X0), p(fc1.W1), p(fc1.W2), p(fc1.b),
                                                        dy.ACT_GELU, p(fc1.Y), p(fc1.H), sp)),
            ("gemm", fc2.flops, lambda: lib.dyad_forward(V, fc2.n_in, fc2.n_out, D, M, dy.BF16,
                                                        p(fc1.Y), p(fc2.W1), p(fc2.W2), p(fc2.b),
                                                        dy.ACT_NONE, p(fc2.Y), None, sp)),
            ("gemm", fc2.flops, lambda: lib.dyad_backward_dx(V, fc2.n_in, fc2.n_out, D, M, dy.BF16,
                                                            p(fc2.dZ0), p(fc2.W1), p(fc2.W2),
                                                            dy.ACT_GELU, p(fc1.H), p(fc2.dX), sp)),
            ("dw", fc2.flops, lambda: lib.dyad_backward_dw(V, fc2.n_in, fc2.n_out, D, M, dy.BF16,
                                                          p(fc2.dZ0), p(fc1.Y), p(fc2.dW1),
                                                          p(fc2.dW2), p(fc2.db), p(ws), ws_bytes, sp)),
            ("gemm", fc1.flops, lambda: lib.dyad_backward_dx(V, fc1.n_in, fc1.n_out, D, M, dy.BF16,
                                                            p(fc2.dX), p(fc1.W1), p(fc1.W2),
                                                            dy.ACT_NONE, None, p(fc1.dX), sp)),
            ("dw", fc1.flops, lambda: lib.dyad_backward_dw(V, fc1.n_in, fc1.n_out, D, M, dy.BF16,
                                                          p(fc2.dX), p(fc1.X0), p(fc1.dW1),
                                                          p(fc1.dW2), p(fc1.db), p(ws), ws_bytes, sp)),
        ]

    step_calls = [(v, c) for v in variants for c in calls(v)]
    flops_step = sum(c[1] for _, c in step_calls)

    def step():
        for _, (_, _, fn) in step_calls:
            check(fn())

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K steps, events on the launch stream only at its ends
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record(stream)
    for _ in range(args.steps):
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_time(t1) / args.steps
    tflops = flops_step / (ms_step * 1e-3) / 1e12

    # per-launch durations: the same K steps again, an event pair around every call
    per = {}
    evs = []
    for _ in range(args.steps):
        for v, (kind, fl, fn) in step_calls:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            check(fn())
            b.record(stream)
            evs.append((v, kind, fl, a, b))
    torch.cuda.synchronize()
    for v, kind, fl, a, b in evs:
        d = per.setdefault(kind, {"ms": 0.0, "n": 0, "flops": 0.0})
        d["ms"] += a.elapsed_time(b)
        d["n"] += 1
        d["flops"] += fl
        dv = per.setdefault(f"{v}", {"ms": 0.0, "n": 0, "flops": 0.0})
        dv["ms"] += a.elapsed_time(b)
        dv["n"] += 1
        dv["flops"] += fl
    dom = max(("gemm", "dw"), key=lambda k: per[k]["ms"])
    avg_ms = per[dom]["ms"] / per[dom]["n"]
    fl_launch = per[dom]["flops"] / per[dom]["n"]
    achieved = fl_launch / (avg_ms * 1e-3) / 1e12
    per_variant = {v: round(per[v]["flops"] / (per[v]["ms"] * 1e-3) / 1e12, 1) for v in variants}

    # dense baseline: same shapes through torch (hipBLASLt), fwd + dX + dW per layer
    dense = None
    if not args.no_dense:
        xs = {}
        for L in (fc1, fc2):
            xs[L] = (torch.randn((L.n_out, L.n_in), device=dev).mul_(0.02).to(torch.bfloat16),
                     torch.randn((M, L.n_in), device=dev).to(torch.bfloat16),
                     torch.randn((M, L.n_out), device=dev).to(torch.bfloat16))

        def dense_ff():
            for L in (fc1, fc2):
                Wd, Xd, dZd = xs[L]
                torch.addmm(L.b, Xd, Wd.t())
                torch.mm(dZd, Wd)
                torch.mm(dZd.t(), Xd)
                dZd.sum(0)
        for _ in range(args.warmup):
            dense_ff()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            dense_ff()
        e1.record(stream)
        torch.cuda.synchronize()
        dense_ms = e0.elapsed_time(e1) / args.steps
        dyad_ms_per_variant = {v: per[v]["ms"] / args.steps for v in variants}
        dense_flops = sum(3 * 2.0 * M * L.n_in * L.n_out for L in (fc1, fc2))
        dense = {"ms_per_ff_fwd_bwd": round(dense_ms, 4),
                 "tflops": round(dense_flops / (dense_ms * 1e-3) / 1e12, 1),
                 "speedup": {v: round(dense_ms / dyad_ms_per_variant[v], 3) for v in variants}}

    # CPU oracle on a bounded token sample (reported baseline only)
    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(wl, args.cpu_tokens)

    traffic = read_traffic(dom, args.workload)
    out = {
        "metric": "Dyad fwd+bwd TFLOP/s and % bf16 MFMA peak; speedup vs dense GEMM, same shape",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "description": wl.note, "n_dyad": D, "tokens": M,
                   "layers": [list(l) for l in wl.layers], "variants": variants,
                   "step": "per variant: fc1 fwd(GELU)+fc2 fwd+fc2 dX(GELU')+fc2 dW+fc1 dX+fc1 dW"},
        "pct_bf16_peak": round(100.0 * tflops / PEAK_BF16_TFLOPS, 2),
        "tflops_per_variant": per_variant,
        "speedup_vs_dense": dense["speedup"] if dense else None,
        "dense": dense,
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "avg_launch_us": round(avg_ms * 1e3, 2),
                     "flops_per_launch": fl_launch, "traffic": traffic},
        "cpu_baseline": cpu,
        "wall_s_timed": round(wall, 3),
    }
    print(json.dumps(out))


def cpu_baseline(wl, tokens):
    """The oracle, as is, on the first `tokens` tokens of the same workload (Dyad-IT)."""
    import numpy as np  # noqa: F401
    import oracle
    from workloads import layer_inputs
    D = wl.n_dyad
    Ms = min(tokens, wl.M)
    flops = 0.0
    t0 = time.perf_counter()
    for li, (_, n_in, n_out) in enumerate(wl.layers):
        L = layer_inputs(n_in, n_out, D, Ms, "bf16", seed_offset=li)
        X, W1, W2, dZ = L.f64("X"), L.f64("W1"), L.f64("W2"), L.f64("dZ")
        oracle.forward("IT", n_in, n_out, D, X, W1, W2, L.f64("bias"))
        oracle.backward_dx("IT", n_in, n_out, D, dZ, W1, W2)
        oracle.backward_dw("IT", n_in, n_out, D, dZ, X)
        flops += 3 * 4.0 * Ms * n_in * n_out / D
    dt = time.perf_counter() - t0
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.threads(),
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": f"{wl.name}, Dyad-IT, every layer fwd+dX+dW+db on {Ms} of {wl.M} tokens "
                      f"(fp64 plain loops, OpenMP)"}


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2312_06881_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def read_traffic(kernel, wl_name):
    """HBM bytes per launch from a committed rocprofv3 --pmc summary, if it matches these sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{wl_name}.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("bytes_per_launch")


if __name__ == "__main__":
    main()
