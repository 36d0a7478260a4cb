#!/usr/bin/env python3
"""Benchmark of the structurally sparsified LSTM backward pass on one MI355X.

One step = the backward pass through time of every layer of the workload
(top layer first; a layer's input gradient is the upstream gradient of the
layer below) with coarse structural sparsifying at the workload's sparsity.
The forward caches are computed once before timing; inputs stay resident in
HBM.  The same step is timed with the dense backward (the speedup
denominator), and a third pass with per-kernel HIP events (recorded on the
launch stream by the library) gives each kernel's average launch duration
for the roofline figure.

Prints ONE JSON line.  value = effective TFLOP/s: the dense backward's flops
(16 H B (I+H) T per layer) divided by the sparse step time.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "LSTM backward ms/step and effective TFLOP/s at 50% structured sparsity vs dense"
DEFAULT_WORKLOAD = "lstm2_lm_h650_b20_t35_f32"
PEAK = {"hbm_gbs": 8000.0, "f32_tflops": 157.3, "bf16_tflops": 2516.6}


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--sparsity", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sparse-only", action="store_true",
                    help="time only the sparse step (for profiler runs)")
    return ap.parse_args()


def kernel_work(wl, layer, Kp, es):
    """Algorithmic bytes and flops of each backward kernel kind for one layer
    call (all T steps): what the method must read and write, not what the
    implementation's staging (split-K partials, chunked updates) adds."""
    I, H, B, T = wl.layer_input(layer), wl.hidden, wl.batch, wl.steps
    K, HB = I + H, H * B
    return {
        # per step: gates_t (4HB, storage type); c_t, c_{t-1}, dH_up[t],
        # dh_rec, dc_t read and dc_{t-1} written (fp32); kept rows and index
        # written
        "gates_select_compact": {"bytes": T * (4 * HB * es + 6 * HB * 4 + Kp * B * es
                                               + Kp // wl.P * 4), "flops": 0},
        # per step: W_c (K' x (I+H)), dG_c (K' x B) read, [dx; dh] ((I+H) x B,
        # fp32) written
        "data_grad_gemm": {"bytes": T * (Kp * K * es + Kp * B * es + K * B * 4),
                           "flops": T * 2 * K * B * Kp},
        # every step's dG_c and [x; h] read once, dW (4H x (I+H), fp32)
        # written once
        "weight_grad_gemm": {"bytes": T * (Kp * B * es + K * B * es) + 4 * H * K * 4,
                             "flops": T * 2 * Kp * K * B},
    }


def roofline_entry(name, work, avg_s, dtype):
    """work: algorithmic bytes/flops of one average launch; avg_s: its mean
    event-measured duration."""
    peak_tf = PEAK["bf16_tflops"] if dtype == "bf16" else PEAK["f32_tflops"]
    t_mem = work["bytes"] / (PEAK["hbm_gbs"] * 1e9)
    t_mfma = work["flops"] / (peak_tf * 1e12)
    if t_mfma > t_mem:
        ach = work["flops"] / avg_s / 1e12
        return {"kernel": name, "bound": "mfma", "achieved": round(ach, 3), "peak": peak_tf,
                "unit": "TFLOP/s", "frac": round(ach / peak_tf, 4), "traffic": None,
                "avg_launch_us": round(avg_s * 1e6, 3), "algorithmic_flops": work["flops"],
                "algorithmic_bytes": work["bytes"]}
    ach = work["bytes"] / avg_s / 1e9
    return {"kernel": name, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK["hbm_gbs"],
            "unit": "GB/s", "frac": round(ach / PEAK["hbm_gbs"], 4), "traffic": None,
            "avg_launch_us": round(avg_s * 1e6, 3), "algorithmic_flops": work["flops"],
            "algorithmic_bytes": work["bytes"]}


def cpu_baseline(wl, inp, sparsity, budget_s=25.0):
    """Time the CPU oracle (as it stands) on a bounded sample of the workload."""
    import oracle
    S = int(round(sparsity * wl.R))
    # sample: the bottom layer's backward over the first T' steps, T' chosen
    # so that one pass is about budget_s of work (estimated from a 1-step probe)
    layer = 0
    I, H, B = wl.layer_input(layer), wl.hidden, wl.batch
    x = inp["x"]
    W = inp["Ws"][layer]
    dH = inp["dH_up"]

    def run(Tp):
        gates, c, h = oracle.forward(x[:Tp], W)
        t0 = time.perf_counter()
        oracle.backward(x[:Tp], W, gates, c, h, dH[:Tp], P=wl.P, R=wl.R, S=S)
        return time.perf_counter() - t0

    t1 = run(1)
    Tp = int(max(1, min(wl.steps, budget_s / max(t1, 1e-6))))
    dt = run(Tp) if Tp > 1 else t1
    flops = 16.0 * H * B * (I + H) * Tp
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": oracle.threads(),
            "kind": "oracle",
            "sample": "fp64 oracle backward (sparsity %.2f) of layer %d over %d of %d steps, "
                      "%.2f s; effective TFLOP/s counts the dense flops 16*H*B*(I+H)*T'"
                      % (sparsity, layer + 1, Tp, wl.steps, dt)}


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only (--gpus 1); multi-GPU sharding is "
              "described in DESIGN.md but not built", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_1806_00512_amd.lstmss as L
    from paper_1806_00512_amd.inputs import WORKLOADS, make_inputs

    wl = WORKLOADS[args.workload]
    sparsity = wl.sparsity if args.sparsity is None else args.sparsity
    dev = torch.device("cuda:0")
    st = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    es = 2 if wl.dtype == "bf16" else 4
    L.load()

    inp = make_inputs(wl, seed=0)
    Ws = [torch.from_numpy(w).to(dev).to(st) for w in inp["Ws"]]
    x0 = torch.from_numpy(inp["x"]).to(dev).to(st)
    dH = torch.from_numpy(inp["dH_up"]).to(dev)

    # forward caches (untimed support for the backward pass)
    xs, caches = [], []
    inp_l = x0
    for li in range(wl.layers):
        h_out, cache = L.fwd_cache(inp_l, Ws[li])
        xs.append(inp_l)
        caches.append(cache)
        inp_l = h_out
    torch.cuda.synchronize()

    def buffers(sp):
        bufs = []
        for li in range(wl.layers):
            I = wl.layer_input(li)
            d = L.dims(wl.steps, wl.batch, I, wl.hidden, st)
            s = L.structure(wl.P, wl.R) if sp > 0 else None
            ws = torch.empty(L.workspace_bytes(d, sp, s), dtype=torch.uint8, device=dev)
            out = {"dX": torch.empty((wl.steps, I, wl.batch), device=dev),
                   "dW": torch.empty((4 * wl.hidden, I + wl.hidden), device=dev),
                   "db": torch.empty(4 * wl.hidden, device=dev),
                   "dh0": torch.empty((wl.hidden, wl.batch), device=dev),
                   "dc0": torch.empty((wl.hidden, wl.batch), device=dev)}
            if sp > 0:
                kp = L.kept_rows(d, sp, s)
                out["idx"] = torch.empty((wl.steps, kp // wl.P), dtype=torch.int32, device=dev)
            bufs.append((ws, out))
        return bufs

    sp_bufs = buffers(sparsity)
    dn_bufs = buffers(0.0)

    def step(sparse):
        up = dH
        for li in reversed(range(wl.layers)):
            if sparse:
                ws, out = sp_bufs[li]
                o = L.bwd_structsparse(xs[li], Ws[li], caches[li], up, sparsity=sparsity, P=wl.P,
                                       R=wl.R, out=out, ws=ws)
            else:
                ws, out = dn_bufs[li]
                o = L.bwd_dense(xs[li], Ws[li], caches[li], up, out=out, ws=ws)
            up = o["dX"]

    def timed(sparse, K, W):
        for _ in range(W):
            step(sparse)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        w0 = time.perf_counter()
        e0.record()
        for _ in range(K):
            step(sparse)
        e1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        return e0.elapsed_time(e1) / K, wall / K * 1e3

    sp_ms, sp_wall = timed(True, args.steps, args.warmup)
    print("sparse: %.4f ms/step (wall %.4f)" % (sp_ms, sp_wall), file=sys.stderr, flush=True)
    if args.sparse_only:
        return
    dn_ms, dn_wall = timed(False, args.steps, args.warmup)
    print("dense: %.4f ms/step (wall %.4f)" % (dn_ms, dn_wall), file=sys.stderr, flush=True)

    # per-kernel HIP-event timing pass (same K sparse steps)
    L.timing_reset()
    L.timing_enable(True)
    for _ in range(args.steps):
        step(True)
    torch.cuda.synchronize()
    kt = L.timing_read()
    L.timing_enable(False)
    L.timing_reset()

    dense_flops = sum(16.0 * wl.hidden * wl.batch * (wl.layer_input(l) + wl.hidden) * wl.steps
                      for l in range(wl.layers))
    sp_kps = []
    for l in range(wl.layers):
        d = L.dims(wl.steps, wl.batch, wl.layer_input(l), wl.hidden, st)
        sp_kps.append(L.kept_rows(d, sparsity, L.structure(wl.P, wl.R)))
    exec_flops = sum(16.0 * wl.hidden * wl.batch * (wl.layer_input(l) + wl.hidden) * wl.steps
                     * sp_kps[l] / (4 * wl.hidden) for l in range(wl.layers))

    # roofline of every kernel kind (work averaged over layers), dominant first
    kernels = {}
    for name in ("gates_select_compact", "data_grad_gemm", "weight_grad_gemm", "aux"):
        ms, n = kt[name]
        kernels[name] = {"total_ms_per_step": round(ms / args.steps, 5), "launches": n,
                         "avg_us": round(ms / max(n, 1) * 1e3, 3)}
    roofs = {}
    for name in ("gates_select_compact", "data_grad_gemm", "weight_grad_gemm"):
        ms, n = kt[name]
        # work of one step (all layers) times the timed steps, spread over
        # the launches of this kind: the average launch's algorithmic work
        works = [kernel_work(wl, l, sp_kps[l], es)[name] for l in range(wl.layers)]
        per_launch = {k: sum(w[k] for w in works) * args.steps / max(n, 1)
                      for k in ("bytes", "flops")}
        roofs[name] = roofline_entry(name, per_launch, ms / 1e3 / max(n, 1), wl.dtype)
    dominant = max(roofs, key=lambda k: kt[k][0])

    result = {
        "metric": METRIC,
        "value": round(dense_flops / (sp_ms / 1e3) / 1e12, 4),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(sp_ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": wl.layers, "input_size": wl.input_size,
                   "hidden": wl.hidden, "batch": wl.batch, "seq_len": wl.steps,
                   "sparsity": sparsity, "P": wl.P, "R": wl.R,
                   "S": int(round(sparsity * wl.R)), "storage": wl.dtype},
        "dense_ms_per_step": round(dn_ms, 5),
        "speedup_vs_dense": round(dn_ms / sp_ms, 4),
        "algorithmic_tflops": round(exec_flops / (sp_ms / 1e3) / 1e12, 4),
        "dense_tflops": round(dense_flops / (dn_ms / 1e3) / 1e12, 4),
        "wall_ms_per_step": {"sparse": round(sp_wall, 5), "dense": round(dn_wall, 5)},
        "kernels": kernels,
        "roofline": roofs[dominant],
        "roofline_all": roofs,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, inp, sparsity)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
