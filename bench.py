"""Benchmark: the Dyad feed-forward block, forward and backward, on one MI355X.

One step = for each of Dyad-IT, -OT and -DT, the feed-forward block of the
chosen workload (default: OPT-125m shapes, fc1 768->3072 with GELU, fc2
3072->768, n_dyad=4, M=16384 tokens, bf16 with fp32 accumulation) run forward
and backward through libdyad's C-ABI: fc1 forward (GELU, pre-activation
stashed), fc2 forward, fc2 input gradient (GELU' fused), fc2 weight+bias
gradient, fc1 input gradient, fc1 weight+bias gradient.  FLOPs are counted
algorithmically, 4*M*n_in*n_out/n_dyad per pass.

Prints one JSON line.  Inputs are seeded synthetic tensors already resident in
HBM when the timed region starts.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
RIDGE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)   # FLOP per byte
METRIC = "Dyad fwd+bwd TFLOP/s and % bf16 MFMA peak; speedup vs dense GEMM, same shape"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="opt125m_ff",
                    help="opt125m_ff (default), opt350m_ff, sweep_d{1024,2048,4096,8192}_D{2,4,8,16}, "
                         "wide_M{16,256,32768}, opt125m_ff_D{3,5,6} (n_dyad 5: zero-padded blocks), tiny_it_f32")
    ap.add_argument("--variants", default="IT,OT,DT")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=16384)
    ap.add_argument("--only", default="",
                    help="run just this call (e.g. IT:fc1.fwd) --steps times, for counter collection")
    ap.add_argument("--block", default="",
                    help="instead of the layer step: time an OPT-125m-shaped decoder block fwd+bwd "
                         "(dense, Dyad FF only, Dyad everywhere) with this variant (IT/OT/DT)")
    ap.add_argument("--fused", action="store_true",
                    help="feed-forward block with GELU inside fc2's kernels (fc1 writes only its "
                         "pre-activation; dyad_forward_ex / dyad_backward_dw_ex)")
    ap.add_argument("--sets", type=int, default=0,
                    help="buffer sets to rotate (default: enough that a set recurs after ~512 MiB of traffic)")
    ap.add_argument("--summarize-counters", metavar="ROOT",
                    help="turn rocprofv3 --pmc runs of --only CALL (subdirectories <call>_sq, <call>_fetch, "
                         "<call>_write of ROOT, call written with ':' and '.' as '_') into "
                         "profiles/counters_<workload>.txt")
    ap.add_argument("--summarize-pmc", nargs=3, metavar=("CALL", "FETCH_DIR", "WRITE_DIR"),
                    help="turn two rocprofv3 --pmc runs of --only CALL (FETCH_SIZE, WRITE_SIZE) into "
                         "profiles/traffic_<workload>.json")
    return ap.parse_args()


def workload(name):
    import workloads as W
    table = {w.name: w for w in [W.OPT125M, W.OPT350M, W.TINY, *W.SWEEP, *W.WIDE, *W.PADDED]}
    if name not in table:
        raise SystemExit(f"unknown workload {name}; choose from {sorted(table)}")
    return table[name]


def algorithmic_bytes(kind, n_in, n_out, D, M, e=2, gelu=False, stash=False):
    """Bytes one pass must move: its operands and results, each once."""
    w = 2 * n_in * n_out // D
    if kind == "fwd":
        return e * (M * n_in + M * n_out + w + n_out + (M * n_out if stash else 0))
    if kind == "dx":
        return e * (M * n_out + w + M * n_in + (M * n_in if gelu else 0))
    return e * (M * n_out + M * n_in + w + n_out)


class Layer:
    """Device buffers of one Dyad layer, allocated once."""

    def __init__(self, torch, n_in, n_out, D, M, seed_offset, dev):
        from workloads import layer_inputs
        L = layer_inputs(n_in, n_out, D, M, "bf16", seed_offset=seed_offset)
        self.n_in, self.n_out, self.D, self.M = n_in, n_out, D, M
        self.W1, self.W2, self.b = L.W1.to(dev), L.W2.to(dev), L.bias.to(dev)
        self.dW1, self.dW2 = torch.empty_like(self.W1), torch.empty_like(self.W2)
        self.db = torch.empty_like(self.b)
        self.X0 = L.X.to(dev)      # input of the first layer
        self.dZ0 = L.dZ.to(dev)    # upstream gradient of the last layer
        self.Y = torch.empty((M, n_out), dtype=torch.bfloat16, device=dev)
        self.H = torch.empty_like(self.Y)
        self.dX = torch.empty((M, n_in), dtype=torch.bfloat16, device=dev)
        self.flops = 4.0 * M * n_in * n_out / D


def build_calls(dy, lib, wl, fc1, fc2, variants, ws, ws_bytes, sp, fused=False):
    """(name, flops, bytes, fn) for every C-ABI call of one step, in step order.  fused: the
    feed-forward block with GELU inside fc2's kernels -- fc1 writes only its pre-activation
    h, fc2's forward and weight gradient read h and apply GELU as they stage it."""
    D, M = wl.n_dyad, wl.M
    vid = {"IT": dy.IT, "OT": dy.OT, "DT": dy.DT}

    def p(t):
        return None if t is None else t.data_ptr()

    out = []
    for v in variants:
        V = vid[v]
        ab = lambda kind, L, **kw: algorithmic_bytes(kind, L.n_in, L.n_out, D, M, **kw)  # noqa: E731
        if fused:
            out += [
                (f"{v}:fc1.fwd", fc1.flops, ab("fwd", fc1),
                 lambda V=V: lib.dyad_forward(V, fc1.n_in, fc1.n_out, D, M, dy.BF16, p(fc1.X0), p(fc1.W1),
                                              p(fc1.W2), p(fc1.b), dy.ACT_NONE, p(fc1.H), None, sp)),
                (f"{v}:fc2.fwd", fc2.flops, ab("fwd", fc2),
                 lambda V=V: lib.dyad_forward_ex(V, fc2.n_in, fc2.n_out, D, M, dy.BF16, dy.ACT_GELU, p(fc1.H),
                                                 p(fc2.W1), p(fc2.W2), p(fc2.b), dy.ACT_NONE, p(fc2.Y), None, sp)),
                (f"{v}:fc2.dx", fc2.flops, ab("dx", fc2, gelu=True),
                 lambda V=V: lib.dyad_backward_dx(V, fc2.n_in, fc2.n_out, D, M, dy.BF16, p(fc2.dZ0),
                                                  p(fc2.W1), p(fc2.W2), dy.ACT_GELU, p(fc1.H), p(fc2.dX), sp)),
                (f"{v}:fc2.dw", fc2.flops, ab("dw", fc2),
                 lambda V=V: lib.dyad_backward_dw_ex(V, fc2.n_in, fc2.n_out, D, M, dy.BF16, dy.ACT_GELU,
                                                     p(fc2.dZ0), p(fc1.H), p(fc2.dW1), p(fc2.dW2), p(fc2.db),
                                                     p(ws), ws_bytes, sp)),
                (f"{v}:fc1.dx", fc1.flops, ab("dx", fc1),
                 lambda V=V: lib.dyad_backward_dx(V, fc1.n_in, fc1.n_out, D, M, dy.BF16, p(fc2.dX), p(fc1.W1),
                                                  p(fc1.W2), dy.ACT_NONE, None, p(fc1.dX), sp)),
                (f"{v}:fc1.dw", fc1.flops, ab("dw", fc1),
                 lambda V=V: lib.dyad_backward_dw(V, fc1.n_in, fc1.n_out, D, M, dy.BF16, p(fc2.dX), p(fc1.X0),
                                                  p(fc1.dW1), p(fc1.dW2), p(fc1.db), p(ws), ws_bytes, sp)),
            ]
            continue
        out += [
            (f"{v}:fc1.fwd", fc1.flops, ab("fwd", fc1, stash=True),
             lambda V=V: lib.dyad_forward(V, fc1.n_in, fc1.n_out, D, M, dy.BF16, p(fc1.X0), p(fc1.W1),
                                          p(fc1.W2), p(fc1.b), dy.ACT_GELU, p(fc1.Y), p(fc1.H), sp)),
            (f"{v}:fc2.fwd", fc2.flops, ab("fwd", fc2),
             lambda V=V: lib.dyad_forward(V, fc2.n_in, fc2.n_out, D, M, dy.BF16, p(fc1.Y), p(fc2.W1),
                                          p(fc2.W2), p(fc2.b), dy.ACT_NONE, p(fc2.Y), None, sp)),
            (f"{v}:fc2.dx", fc2.flops, ab("dx", fc2, gelu=True),
             lambda V=V: lib.dyad_backward_dx(V, fc2.n_in, fc2.n_out, D, M, dy.BF16, p(fc2.dZ0),
                                              p(fc2.W1), p(fc2.W2), dy.ACT_GELU, p(fc1.H), p(fc2.dX), sp)),
            (f"{v}:fc2.dw", fc2.flops, ab("dw", fc2),
             lambda V=V: lib.dyad_backward_dw(V, fc2.n_in, fc2.n_out, D, M, dy.BF16, p(fc2.dZ0), p(fc1.Y),
                                              p(fc2.dW1), p(fc2.dW2), p(fc2.db), p(ws), ws_bytes, sp)),
            (f"{v}:fc1.dx", fc1.flops, ab("dx", fc1),
             lambda V=V: lib.dyad_backward_dx(V, fc1.n_in, fc1.n_out, D, M, dy.BF16, p(fc2.dX), p(fc1.W1),
                                              p(fc1.W2), dy.ACT_NONE, None, p(fc1.dX), sp)),
            (f"{v}:fc1.dw", fc1.flops, ab("dw", fc1),
             lambda V=V: lib.dyad_backward_dw(V, fc1.n_in, fc1.n_out, D, M, dy.BF16, p(fc2.dX), p(fc1.X0),
                                              p(fc1.dW1), p(fc1.dW2), p(fc1.db), p(ws), ws_bytes, sp)),
        ]
    return out


def block_bench(args):
    """OPT-125m-shaped pre-LN decoder block (d 768, 12 heads, ffn 3072, causal self-attention;
    batch 8 x 2048 tokens) forward + backward on synthetic bf16 tokens, three ways: dense
    nn.Linear everywhere, Dyad in the two FF layers only, Dyad in every linear layer (FF and
    the q / k / v / out projections); plus the FF sub-block alone, dense vs Dyad.  Attention
    scores and softmax run in fp32 through plain matmuls (contiguous operands)."""
    import math
    import torch
    import torch.nn.functional as F
    from paper_2312_06881_amd.nn import DyadFF, DyadLinear

    d, ffn, heads, D, B, T = 768, 3072, 12, 4, 8, 2048
    hd = d // heads
    v = args.block
    dev = torch.device("cuda:0")
    torch.manual_seed(0)
    bf = torch.bfloat16

    def lin(i, o, dyad):
        return DyadLinear(i, o, D, v, device=dev) if dyad else torch.nn.Linear(i, o, device=dev, dtype=bf)

    class DenseFF(torch.nn.Module):
        def __init__(self):
            super().__init__()
            self.fc1, self.fc2 = lin(d, ffn, False), lin(ffn, d, False)

        def forward(self, x):
            return self.fc2(F.gelu(self.fc1(x)))

    mask = torch.full((T, T), float("-inf"), device=dev).triu(1)

    class Block(torch.nn.Module):
        def __init__(self, attn_dyad, ff_dyad):
            super().__init__()
            self.ln1 = torch.nn.LayerNorm(d, device=dev, dtype=bf)
            self.ln2 = torch.nn.LayerNorm(d, device=dev, dtype=bf)
            self.q, self.k, self.v, self.o = (lin(d, d, attn_dyad) for _ in range(4))
            self.ff = DyadFF(d, ffn, D, v, device=dev) if ff_dyad else DenseFF()

        def forward(self, x):
            h = self.ln1(x)
            q, k, w = (t.reshape(B, T, heads, hd).transpose(1, 2).float() for t in (self.q(h), self.k(h), self.v(h)))
            s = torch.matmul(q.contiguous(), k.transpose(-1, -2).contiguous()) / math.sqrt(hd) + mask
            a = torch.matmul(torch.softmax(s, dim=-1), w.contiguous())
            x = x + self.o(a.transpose(1, 2).reshape(B, T, d).to(bf).contiguous())
            return x + self.ff(self.ln2(x))

    x = torch.randn((B, T, d), device=dev, dtype=bf)
    g = torch.randn((B, T, d), device=dev, dtype=bf)

    def timed(mod, inp):
        xi = inp.detach().requires_grad_(True)
        for _ in range(args.warmup):
            mod(xi).backward(g)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            mod(xi).backward(g)
        e1.record()
        torch.cuda.synchronize()
        return round(e0.elapsed_time(e1) / args.steps, 4)

    res = {"dense": timed(Block(False, False), x), "dyad_ff": timed(Block(False, True), x),
           "dyad_all": timed(Block(True, True), x),
           "ff_dense": timed(DenseFF(), x), "ff_dyad": timed(DyadFF(d, ffn, D, v, device=dev), x)}
    print(json.dumps({
        "metric": "decoder block forward+backward ms (OPT-125m shape)", "unit": "ms",
        "higher_is_better": False, "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "opt125m_decoder_block", "d": d, "ffn": ffn, "heads": heads, "n_dyad": D,
                   "variant": v, "batch": B, "seq_len": T},
        "ms": res,
        "speedup_vs_dense": {"block_dyad_ff": round(res["dense"] / res["dyad_ff"], 3),
                             "block_dyad_all": round(res["dense"] / res["dyad_all"], 3),
                             "ff_only": round(res["ff_dense"] / res["ff_dyad"], 3)},
    }))


def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(args, *args.summarize_pmc)
        return
    if args.summarize_counters:
        summarize_counters(args, args.summarize_counters)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "libdyad runs on one GPU; --gpus must be 1 "
                                   "(token sharding over several GPUs is a design, not code)",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.block:
        block_bench(args)
        return
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

    if len(wl.layers) == 2:
        (_, i1, o1), (_, i2, o2) = wl.layers
    else:
        (_, i1, o1), = wl.layers
        i2, o2 = o1, i1
    # Buffer sets, rotated call by call: consecutive calls never touch the same
    # buffers, and a set comes round again only after about 1 GiB of other
    # calls' traffic (four times the 256 MB last-level cache), so small-batch
    # calls read their weights from HBM, not from the cache.
    mean_call = sum(algorithmic_bytes(k, n_in, n_out, D, M) for (_, n_in, n_out) in
                    ((None, i1, o1), (None, i2, o2)) for k in ("fwd", "dx", "dw")) / 6
    n_sets = max(1, min(16, -(-(1 << 30) // int(mean_call))))
    if args.sets:
        n_sets = args.sets
    layers = [(Layer(torch, i1, o1, D, M, 0, dev), Layer(torch, i2, o2, D, M, 1, dev)) for _ in range(n_sets)]
    fc1, fc2 = layers[0]
    ws_bytes = max(dy.dyad_dw_workspace_bytes_ex(vid[v], L.n_in, L.n_out, D, M, dy.BF16, a)
                   for v in variants for L in (fc1, fc2) for a in (dy.ACT_NONE, dy.ACT_GELU))
    ws = torch.empty((max(ws_bytes, 16),), dtype=torch.uint8, device=dev)

    def check(rc):
        if rc != 0:
            raise RuntimeError(dy.dyad_strerror(rc))

    sets = [build_calls(dy, lib, wl, a, b, variants, ws, ws_bytes, sp, args.fused) for a, b in layers]
    calls = sets[0]
    n_calls = len(calls)
    if args.only:
        # counter collection: one call, repeated, plus a plain copy of known size
        idx = [i for i, c in enumerate(calls) if c[0] == args.only]
        if not idx:
            raise SystemExit(f"--only {args.only}: no such call; one of {[c[0] for c in calls]}")
        src = torch.empty((COPY_BYTES,), dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for r in range(args.steps):
            check(sets[r % n_sets][idx[0]][3]())
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"only": args.only, "launches": args.steps, "copy_bytes": src.numel(),
                          "buffer_sets": n_sets, "algorithmic_bytes": calls[idx[0]][2],
                          "flops": calls[idx[0]][1]}))
        return

    flops_step = sum(c[1] for c in calls)
    rot = [0]

    def step():
        # call c of the step takes the next buffer set in turn
        for c in range(n_calls):
            check(sets[rot[0] % n_sets][c][3]())
            rot[0] += 1

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K whole steps between two events on the launch stream
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

    # per-call durations: at least 50 more steps with an event pair around every call
    reps = max(50, args.steps)
    evs = []
    for _ in range(reps):
        for c in range(n_calls):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            call = sets[rot[0] % n_sets][c]
            rot[0] += 1
            a.record(stream)
            check(call[3]())
            b.record(stream)
            evs.append((call, a, b))
    torch.cuda.synchronize()
    per = {}
    for c, a, b in evs:
        d = per.setdefault(c[0], {"t": [], "flops": c[1], "bytes": c[2]})
        d["t"].append(a.elapsed_time(b))
    table = {}
    for name, d in per.items():
        t = sorted(d["t"])
        d["ms"] = sum(t)
        d["n"] = len(t)
        us = d["ms"] / d["n"] * 1e3
        q = lambda f: t[min(len(t) - 1, int(f * (len(t) - 1) + 0.5))] * 1e3  # noqa: E731
        table[name] = {"us": round(us, 2), "us_median": round(q(0.5), 2), "us_p10": round(q(0.1), 2),
                       "us_p90": round(q(0.9), 2), "reps": len(t),
                       "tflops": round(d["flops"] / (q(0.5) * 1e-6) / 1e12, 1),
                       "gbs": round(d["bytes"] / (q(0.5) * 1e-6) / 1e9, 1),
                       "bound": "hbm" if d["flops"] / d["bytes"] < RIDGE else "mfma"}
    dom = max(per, key=lambda n: per[n]["ms"])
    dd = per[dom]
    avg_s = dd["ms"] / dd["n"] * 1e-3
    if table[dom]["bound"] == "hbm":
        achieved, peak, unit = dd["bytes"] / avg_s / 1e9, PEAK_HBM_GBS, "GB/s"
    else:
        achieved, peak, unit = dd["flops"] / avg_s / 1e12, PEAK_BF16_TFLOPS, "TFLOP/s"
    per_variant = {}
    for v in variants:
        ms_v = sum(per[n]["ms"] / per[n]["n"] for n in per if n.startswith(v + ":"))
        fl_v = sum(per[n]["flops"] for n in per if n.startswith(v + ":"))
        per_variant[v] = {"ms": round(ms_v, 4), "tflops": round(fl_v / (ms_v * 1e-3) / 1e12, 1)}

    dense = None
    if not args.no_dense:
        dense = dense_baseline(torch, fc1, fc2, M, dev, stream, args)
        dense["speedup"] = {v: round(dense["ms_per_ff_fwd_bwd"] / per_variant[v]["ms"], 3)
                            for v in variants}

    cpu = None if args.no_cpu else cpu_baseline(wl, args.cpu_tokens)

    out = {
        "metric": METRIC,
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
                   "step": ("per variant: fc1 fwd (pre-activation only) + fc2 fwd (GELU on load) + "
                            "fc2 dX(GELU') + fc2 dW+db (GELU on load) + fc1 dX + fc1 dW+db") if args.fused else
                           ("per variant: fc1 fwd(GELU, stash) + fc2 fwd + fc2 dX(GELU') + fc2 dW+db "
                            "+ fc1 dX + fc1 dW+db"),
                   "fused_ff": bool(args.fused),
                   "buffer_sets": n_sets},
        "pct_bf16_peak": round(100.0 * tflops / PEAK_BF16_TFLOPS, 2),
        "per_variant": per_variant,
        "speedup_vs_dense": dense["speedup"] if dense else None,
        "dense": dense,
        "roofline": {"bound": table[dom]["bound"], "call": dom, "achieved": round(achieved, 1),
                     "peak": peak, "unit": unit, "frac": round(achieved / peak, 4),
                     "avg_launch_us": round(avg_s * 1e6, 2), "median_launch_us": table[dom]["us_median"],
                     "flops_per_launch": dd["flops"],
                     "bytes_per_launch": dd["bytes"],
                     "traffic": read_traffic(dom, wl.name)},
        "per_call": table,
        "cpu_baseline": cpu,
        "wall_s_timed": round(wall, 3),
    }
    print(json.dumps(out))


def dense_baseline(torch, fc1, fc2, M, dev, stream, args):
    """Same-shape dense layers through torch (hipBLASLt): fwd X W^T + b, dX = dZ W, dW = dZ^T X, db."""
    xs = {}
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    for L in (fc1, fc2):
        xs[L] = (torch.randn((L.n_out, L.n_in), device=dev, generator=g).mul_(0.02).to(torch.bfloat16),
                 torch.randn((M, L.n_in), device=dev, generator=g).to(torch.bfloat16),
                 torch.randn((M, L.n_out), device=dev, generator=g).to(torch.bfloat16))

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
    ms = e0.elapsed_time(e1) / args.steps
    flops = sum(3 * 2.0 * M * L.n_in * L.n_out for L in (fc1, fc2))
    return {"ms_per_ff_fwd_bwd": round(ms, 4), "tflops": round(flops / (ms * 1e-3) / 1e12, 1)}


def cpu_baseline(wl, tokens):
    """The oracle, as it stands, on the first `tokens` tokens of the same workload (Dyad-IT).
    The inputs are drawn before the clock starts; only the oracle's passes are timed."""
    import oracle
    from workloads import layer_inputs
    D = wl.n_dyad
    Ms = min(tokens, wl.M)
    inputs = []
    for li, (_, n_in, n_out) in enumerate(wl.layers):
        L = layer_inputs(n_in, n_out, D, Ms, "bf16", seed_offset=li)
        inputs.append((n_in, n_out, L.f64("X"), L.f64("W1"), L.f64("W2"), L.f64("dZ"), L.f64("bias")))
    flops = 0.0
    t0 = time.perf_counter()
    for n_in, n_out, X, W1, W2, dZ, b in inputs:
        oracle.forward("IT", n_in, n_out, D, X, W1, W2, b)
        oracle.backward_dx("IT", n_in, n_out, D, dZ, W1, W2)
        oracle.backward_dw("IT", n_in, n_out, D, dZ, X)
        flops += 3 * 4.0 * Ms * n_in * n_out / D
    dt = time.perf_counter() - t0
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.threads(),
            "kind": "oracle", "seconds": round(dt, 2),
            "sample": f"{wl.name}, Dyad-IT only, every layer fwd + dX + dW + db on {Ms} of {wl.M} "
                      f"tokens (fp64 plain loops, OpenMP); inputs drawn before the timer"}


COPY_BYTES = 256 << 20   # the plain copy --only runs beside the call, for counter calibration


def _pmc_rows(run_dir):
    import csv
    import glob
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    return list(csv.DictReader(open(files[0])))


def _per_launch(rows, counter):
    """(average KiB per launch of the call's kernels, KiB the copy kernel read/wrote, launches)."""
    rows = [r for r in rows if r["Counter_Name"] == counter]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    copies = [r for r in rows if "copyBuffer" in r["Kernel_Name"]]
    big = max(int(r["Grid_Size"]) for r in copies)
    copy_kib = [float(r["Counter_Value"]) for r in copies if int(r["Grid_Size"]) == big]
    # the call's kernels sit between consecutive copies: one launch = the dispatches of one gap
    launches, cur = [], 0.0
    for r in rows:
        if "copyBuffer" in r["Kernel_Name"]:
            if int(r["Grid_Size"]) == big and cur > 0:
                launches.append(cur)
                cur = 0.0
        else:
            cur += float(r["Counter_Value"])
    if cur > 0:
        launches.append(cur)
    return sum(launches) / len(launches), sum(copy_kib) / len(copy_kib), len(launches)


def summarize_pmc(args, call, fetch_dir, write_dir):
    """HBM bytes per launch of `call`: FETCH_SIZE and WRITE_SIZE (KiB per dispatch), each scaled by
    what the same counter reads for a plain 256 MiB copy run beside it."""
    f_kib, f_copy, n_f = _per_launch(_pmc_rows(fetch_dir), "FETCH_SIZE")
    w_kib, w_copy, n_w = _per_launch(_pmc_rows(write_dir), "WRITE_SIZE")
    f_scale = COPY_BYTES / (f_copy * 1024)
    w_scale = COPY_BYTES / (w_copy * 1024)
    fetch = f_kib * 1024 * f_scale
    write = w_kib * 1024 * w_scale
    path = os.path.join(ROOT, "profiles", f"traffic_{args.workload}.json")
    wl = "" if args.workload == "opt125m_ff" else f" --workload {args.workload}"
    rec = {}
    if os.path.exists(path):
        rec = json.load(open(path))
    if rec.get("source_hash") != kernel_source_hash():
        rec = {"source_hash": kernel_source_hash(), "calls": {}}
    rec["calls"][call] = {"hbm_bytes_per_launch": round(fetch + write), "fetch_bytes": round(fetch),
                          "write_bytes": round(write), "fetch_raw_kib": round(f_kib, 1),
                          "write_raw_kib": round(w_kib, 1), "fetch_scale": round(f_scale, 4),
                          "write_scale": round(w_scale, 4), "launches": [n_f, n_w],
                          "commands": [f"rocprofv3 --pmc {c} --output-format csv -d <dir>/{c} -o run -- "
                                       f"python -u bench.py{wl} --only {call} --steps 5" for c in ("FETCH_SIZE", "WRITE_SIZE")]
                          + [f"python bench.py{wl} --summarize-pmc {call} <dir>/FETCH_SIZE <dir>/WRITE_SIZE"]}
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w") as fh:
        json.dump(rec, fh, indent=1, sort_keys=True)
    print(json.dumps({call: rec["calls"][call]}))


SQ_COUNTERS = ("SQ_WAVES SQ_BUSY_CYCLES SQ_WAVE_CYCLES SQ_WAIT_INST_ANY SQ_VALU_MFMA_BUSY_CYCLES "
               "SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_BUSY_CU_CYCLES GRBM_GUI_ACTIVE")
N_SIMD, N_XCD = 1024, 8   # MI355X: 256 CUs x 4 SIMDs, in 8 XCDs


def _kernel_short(name):
    """A kernel's name without its argument list and return type (keeps '(anonymous namespace)')."""
    name = name.strip()
    if name.endswith(")"):
        depth = 0
        for i in range(len(name) - 1, -1, -1):
            depth += {")": 1, "(": -1}.get(name[i], 0)
            if depth == 0:
                name = name[:i]
                break
    return name[5:] if name.startswith("void ") else name


def _launch_sums(rows, counters):
    """Per launch of the call (its kernels between two copies): counter sums, and the copy's values."""
    rows = sorted(rows, key=lambda r: int(r["Dispatch_Id"]))
    copies = [r for r in rows if "copyBuffer" in r["Kernel_Name"]]
    big = max(int(r["Grid_Size"]) for r in copies) if copies else 0
    launches, cur, kernels = [], {}, set()
    for r in rows:
        if "copyBuffer" in r["Kernel_Name"]:
            if int(r["Grid_Size"]) == big and cur:
                launches.append(cur)
                cur = {}
            continue
        if r["Counter_Name"] in counters:
            cur[r["Counter_Name"]] = cur.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
            kernels.add(_kernel_short(r["Kernel_Name"]))
    if cur:
        launches.append(cur)
    copy = {}
    for r in copies:
        if int(r["Grid_Size"]) == big:
            copy.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    return launches, {k: sum(v) / len(v) for k, v in copy.items()}, sorted(kernels)


def summarize_counters(args, root):
    """One row per call: MFMA utilisation (SQ_VALU_MFMA_BUSY_CYCLES over N_SIMD x the GPU's active
    cycles per XCD), waves' share of cycles waiting (SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES), achieved
    TFLOP/s from the counted MFMA work (512 FLOP per MOPS unit), and HBM bytes per launch
    (FETCH_SIZE / WRITE_SIZE scaled by the same counters of a plain copy of known size)."""
    import glob
    lines = []
    for sq_dir in sorted(glob.glob(os.path.join(root, "*_sq"))):
        tag = os.path.basename(sq_dir)[:-3]
        call = tag.replace("_fc", ":fc").replace("_fwd", ".fwd").replace("_dx", ".dx").replace("_dw", ".dw")
        sq, _, kernels = _launch_sums(_pmc_rows(sq_dir), SQ_COUNTERS.split())
        avg = {k: sum(l.get(k, 0.0) for l in sq) / len(sq) for k in SQ_COUNTERS.split()}
        cycles = avg["GRBM_GUI_ACTIVE"] / N_XCD
        mfma = avg["SQ_VALU_MFMA_BUSY_CYCLES"] / (N_SIMD * cycles) if cycles else 0.0
        wait = avg["SQ_WAIT_INST_ANY"] / avg["SQ_WAVE_CYCLES"] if avg["SQ_WAVE_CYCLES"] else 0.0
        flop = avg["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512
        fb = wb = None
        fdir, wdir = os.path.join(root, tag + "_fetch"), os.path.join(root, tag + "_write")
        if os.path.isdir(fdir) and os.path.isdir(wdir):
            fl, fc, _ = _launch_sums(_pmc_rows(fdir), ["FETCH_SIZE"])
            wl, wc, _ = _launch_sums(_pmc_rows(wdir), ["WRITE_SIZE"])
            fb = sum(l["FETCH_SIZE"] for l in fl) / len(fl) * 1024 * COPY_BYTES / (fc["FETCH_SIZE"] * 1024)
            wb = sum(l["WRITE_SIZE"] for l in wl) / len(wl) * 1024 * COPY_BYTES / (wc["WRITE_SIZE"] * 1024)
        lines.append((call, len(sq), cycles, mfma, wait, flop, fb, wb, kernels))
    path = os.path.join(ROOT, "profiles", f"counters_{args.workload}.txt")
    with open(path, "w") as fh:
        fh.write(f"# Hardware counters per launch, workload {args.workload} (one MI355X, bf16), "
                 f"kernel sources {kernel_source_hash()}.\n"
                 f"# commands, per call C (tag T = C with ':' and '.' as '_'), each its own run:\n"
                 f"#   rocprofv3 --pmc {SQ_COUNTERS} --output-format csv -d <root>/T_sq -o run -- "
                 f"python -u bench.py --workload {args.workload} --only C --steps 5\n"
                 f"#   rocprofv3 --pmc FETCH_SIZE ... -d <root>/T_fetch ...;  rocprofv3 --pmc WRITE_SIZE ... "
                 f"-d <root>/T_write ...\n"
                 f"#   python bench.py --workload {args.workload} --summarize-counters <root>\n"
                 f"# mfma_util = SQ_VALU_MFMA_BUSY_CYCLES / ({N_SIMD} SIMDs x GRBM_GUI_ACTIVE / {N_XCD} XCDs);"
                 f" wait = SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES;\n"
                 f"# mfma_flop = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512; HBM bytes = FETCH_SIZE / WRITE_SIZE scaled by "
                 f"what they read for a plain {COPY_BYTES >> 20} MiB copy in the same run.\n"
                 f"{'call':12s} {'launches':>8s} {'cycles/XCD':>11s} {'mfma_util':>9s} {'wait':>6s} "
                 f"{'mfma_GFLOP':>10s} {'fetch_MB':>9s} {'write_MB':>9s}  kernels\n")
        for call, n, cyc, mf, wt, fl, fb, wb, ks in lines:
            fh.write(f"{call:12s} {n:8d} {cyc:11.0f} {mf:9.3f} {wt:6.3f} {fl / 1e9:10.2f} "
                     f"{'-' if fb is None else f'{fb / 1e6:9.1f}':>9s} {'-' if wb is None else f'{wb / 1e6:9.1f}':>9s}  "
                     f"{'; '.join(k.replace('dyad::', '').replace('(anonymous namespace)::', '') for k in ks)}\n")
    print(open(path).read())


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2312_06881_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def read_traffic(call, wl_name):
    """HBM bytes per launch of `call` from a committed counter summary, if it matches these sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{wl_name}.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("calls", {}).get(call, {}).get("hbm_bytes_per_launch")


if __name__ == "__main__":
    main()
