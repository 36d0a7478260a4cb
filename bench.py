#!/usr/bin/env python3
"""Benchmark of the structurally sparsified LSTM backward pass on one MI355X.

One step = the backward pass through time of every layer of the workload
(a layer's input gradient is the upstream gradient of the layer below) with
coarse structural sparsifying at the workload's sparsity, run as one
wavefront stack call (lstm_bwd_stack: the layers overlap in time, each
lagging the one above by one input-gradient launch).  The forward caches are
computed once before timing; inputs stay resident in HBM.  The same step is
timed with the dense backward (the speedup denominator), with the layers
called one after the other, with 9-sparse : 1-dense and 3 : 1 schedules, and
a last pass of single-layer calls with per-kernel HIP events (recorded on
each kernel's launch stream by the library) gives each kernel's average
launch duration for the roofline.  The forward pass, whole training steps
(dense-after-sparse trainer) and the fine-grained structure are timed
beside it.

Default workload: the 4-layer sequence-to-sequence encoder shape
(I = H = 2048, B = 128, T = 50, fp32).  Every other workload shape (the
small 1-layer H = 128 case, the 2-layer language-model shape, the 2-layer
H = 1024 shape with its sparsity sweep, and the bf16 1-layer H = 4096 shape
with its 9 sparse : 1 dense schedule) is measured beside it and reported
under "also", each with its own per-kernel roofline.

Prints ONE JSON line.  value = effective TFLOP/s: the dense backward's flops
(16 H B (I+H) T per layer) divided by the sparse step time.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "LSTM backward ms/step and effective TFLOP/s at 50% structured sparsity vs dense"
DEFAULT_WORKLOAD = "lstm4_enc_h2048_b128_t50_f32"
ALSO_WORKLOADS = ("lstm1_h128_b16_t20_f32", "lstm2_lm_h650_b20_t35_f32",
                  "lstm2_h1024_b64_t35_f32", "lstm1_h4096_b256_t100_bf16")
PEAK = {"hbm_gbs": 8000.0, "f32_tflops": 157.3, "bf16_tflops": 2516.6}
KINDS = ("gates_select_compact", "data_grad_gemm", "weight_grad_gemm")
# device kernel behind each timed kind whose HBM counters may be on file
KIND_KERNEL = {"gates_select_compact": "cell", "data_grad_gemm": "gemm1_kernel",
               "weight_grad_gemm": "wgrad_kernel"}
KERNEL_SOURCES = tuple("paper_1806_00512_amd/csrc/" + f for f in (
    "gemm_common.h", "gemm1.hip", "wgrad.h", "wgrad_f32.hip", "wgrad_bf16.hip", "gemm.hip",
    "cell.hip", "select.h", "common.h", "kernels.h", "lstmss_api.cpp"))


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--sparsity", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-also", action="store_true", help="skip the secondary workloads")
    ap.add_argument("--sparse-only", action="store_true",
                    help="time only the sparse step (for profiler runs)")
    ap.add_argument("--serial", action="store_true",
                    help="run the weight/input-gradient work in order on the main stream "
                         "(isolated per-kernel durations) instead of on the side stream")
    ap.add_argument("--no-bidir", action="store_true",
                    help="skip the bidirectional-layer measurement")
    ap.add_argument("--no-train", action="store_true",
                    help="skip the whole-training-step measurement")
    ap.add_argument("--no-fine", action="store_true",
                    help="skip the fine-grained structure measurement")
    ap.add_argument("--fine-my", type=int, default=8, help="fine structure: block width My")
    ap.add_argument("--fine-mx", type=int, default=4, help="fine structure: rows per slice Mx")
    ap.add_argument("--calibration-copy-mib", type=int, default=0,
                    help="first run one device-to-device copy of this many MiB (the known-size "
                         "kernel that scales HBM counter readings)")
    return ap.parse_args()


def kernel_work(wl, layer, Kp, es, select_in_product=False):
    """Algorithmic bytes and flops of each backward kernel kind for one layer
    call (all T steps): what the method must read and write, not what the
    implementation's staging (split-K partials, chunked updates) adds.  The
    kept rows and the offset index are written by the gate kernels, or by
    the dh product when the selection runs inside it (select_in_product)."""
    I, H, B, T = wl.layer_input(layer), wl.hidden, wl.batch, wl.steps
    K, HB = I + H, H * B
    compact = Kp * B * es + Kp // wl.P * 4
    return {
        # per step: gates_t (4HB, storage type); c_t, c_{t-1}, dH_up[t],
        # dh_rec, dc_t read and dc_{t-1} written (fp32); kept rows and index
        # written (unless the dh product writes them)
        "gates_select_compact": {"bytes": T * (4 * HB * es + 6 * HB * 4
                                               + (0 if select_in_product else compact)),
                                 "flops": 0},
        # per step: W_c (K' x (I+H)), dG_c (K' x B) read, [dx; dh] ((I+H) x B,
        # fp32) written; kept rows and index written when it selects
        "data_grad_gemm": {"bytes": T * (Kp * K * es + Kp * B * es + K * B * 4
                                         + (compact if select_in_product else 0)),
                           "flops": T * 2 * K * B * Kp},
        # every step's dG_c and [x; h] read once, dW (4H x (I+H), fp32)
        # written once
        "weight_grad_gemm": {"bytes": T * (Kp * B * es + K * B * es) + 4 * H * K * 4,
                             "flops": T * 2 * Kp * K * B},
    }


def sources_digest():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_on_file(kind, workload):
    """HBM bytes per launch from the committed counter summary of this kernel
    and workload, or None when there is none or the kernel sources changed
    since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic_%s_%s.txt" % (KIND_KERNEL[kind], workload))
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith((" ", "#")):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    if rec.get("sources_sha256_16") != sources_digest():
        return None
    try:
        return float(rec["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def rocprof_on_file(kind, workload):
    """Average launch duration (us) of a kernel kind in the committed
    rocprofv3 kernel-trace summary of this workload's benchmark command (its
    per-kernel timing pass), or None when there is none or the kernel sources
    changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "kernels_%s.txt" % workload)
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith((" ", "#")):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    if rec.get("sources_sha256_16") != sources_digest():
        return None
    try:
        return float(rec["rocprof_avg_us_" + kind])
    except (KeyError, ValueError):
        return None


def roofline_entry(name, work, avg_s, dtype, traffic, rocprof_us=None):
    """work: algorithmic bytes/flops of one average launch; avg_s: its mean
    event-measured duration; rocprof_us: the same kind's average duration in
    the committed rocprofv3 summary (frac_rocprof is then reported beside
    frac)."""
    peak_tf = PEAK["bf16_tflops"] if dtype == "bf16" else PEAK["f32_tflops"]
    t_mem = work["bytes"] / (PEAK["hbm_gbs"] * 1e9)
    t_mfma = work["flops"] / (peak_tf * 1e12)
    common = {"traffic": None if traffic is None else round(traffic),
              "avg_launch_us": round(avg_s * 1e6, 3), "algorithmic_flops": work["flops"],
              "algorithmic_bytes": work["bytes"]}
    if rocprof_us:
        common["avg_launch_us_rocprof"] = round(rocprof_us, 3)
    if t_mfma > t_mem:
        ach = work["flops"] / avg_s / 1e12
        e = dict({"kernel": name, "bound": "mfma", "achieved": round(ach, 3), "peak": peak_tf,
                  "unit": "TFLOP/s", "frac": round(ach / peak_tf, 4)}, **common)
        if rocprof_us:
            e["frac_rocprof"] = round(work["flops"] / (rocprof_us * 1e-6) / 1e12 / peak_tf, 4)
        return e
    ach = work["bytes"] / avg_s / 1e9
    e = dict({"kernel": name, "bound": "hbm", "achieved": round(ach, 1),
              "peak": PEAK["hbm_gbs"], "unit": "GB/s", "frac": round(ach / PEAK["hbm_gbs"], 4)},
             **common)
    if rocprof_us:
        e["frac_rocprof"] = round(work["bytes"] / (rocprof_us * 1e-6) / 1e9 / PEAK["hbm_gbs"], 4)
    return e


def roofline_all(L, wl, sparsity, kt, steps):
    """Roofline entry of every timed kernel kind from a per-kernel timing pass
    (kt) of `steps` sparse steps of workload wl."""
    st_dt = "bf16" if wl.dtype == "bf16" else "f32"
    es = 2 if wl.dtype == "bf16" else 4
    dims = [L.dims(wl.steps, wl.batch, wl.layer_input(l), wl.hidden, st_dt)
            for l in range(wl.layers)]
    kps = [L.kept_rows(d, sparsity, L.structure(wl.P, wl.R)) for d in dims]
    sel = [L.bwd_info(d, sparsity, L.structure(wl.P, wl.R))["select_in_product"] for d in dims]
    roofs = {}
    for name in KINDS:
        ms, n = kt[name]
        # work of one step (all layers) times the timed steps, spread over
        # the launches of this kind: the average launch's algorithmic work
        works = [kernel_work(wl, l, kps[l], es, sel[l])[name] for l in range(wl.layers)]
        per_launch = {k: sum(w[k] for w in works) * steps / max(n, 1) for k in ("bytes", "flops")}
        roofs[name] = roofline_entry(name, per_launch, ms / 1e3 / max(n, 1), wl.dtype,
                                     traffic_on_file(name, wl.name),
                                     rocprof_on_file(name, wl.name))
        roofs[name]["select_in_product"] = any(sel)
    return roofs, kps


def kernel_table(kt, steps):
    return {name: {"total_ms_per_step": round(kt[name][0] / steps, 5), "launches": kt[name][1],
                   "avg_us": round(kt[name][0] / max(kt[name][1], 1) * 1e3, 3)}
            for name in KINDS + ("aux",)}


def cpu_baseline(wl, inp, sparsity, budget_s=20.0, budget_1core_s=10.0):
    """Time the CPU oracle (as it stands) on a bounded sample of the workload,
    once with all host cores (the oracle's OpenMP threads) and once on one
    core: the backward of the first T' steps of the bottom layer, T' sized
    from a 2-step probe to about the budget; with all cores, when a whole
    layer is shorter than that, further layers of the same call (each with
    the oracle's own input) are added while the total stays under budget_s."""
    import oracle
    S = int(round(sparsity * wl.R))
    x = inp["x"]
    dH = inp["dH_up"]

    def run(layer_x, W, Tp):
        gates, c, h = oracle.forward(layer_x[:Tp], W)
        t0 = time.perf_counter()
        oracle.backward(layer_x[:Tp], W, gates, c, h, dH[:Tp], P=wl.P, R=wl.R, S=S)
        return time.perf_counter() - t0, h

    def sized(budget):
        Tp = 2
        dt, h = run(x, inp["Ws"][0], Tp)
        for _ in range(3):  # re-size from the last run (the first pays thread start-up)
            want = int(max(2, min(wl.steps, Tp * budget / max(dt, 1e-6))))
            if want <= Tp or (dt >= 0.5 * budget and want < 2 * Tp):
                break
            Tp = want
            dt, h = run(x, inp["Ws"][0], Tp)
        return Tp, dt, h

    def flops(layer, Tp):
        return 16.0 * wl.hidden * wl.batch * (wl.layer_input(layer) + wl.hidden) * Tp

    cores = oracle.threads()
    Tp, dt, h = sized(budget_s)
    fl = flops(0, Tp)
    layers = 1
    while Tp == wl.steps and layers < wl.layers and dt * (layers + 1) / layers <= budget_s:
        d1, h = run(h[1:], inp["Ws"][layers], Tp)
        dt += d1
        fl += flops(layers, Tp)
        layers += 1
    out = {"value": round(fl / dt / 1e12, 6), "unit": "TFLOP/s", "cores": cores,
           "kind": "oracle",
           "sample": "fp64 oracle backward (sparsity %.2f) of the bottom %d layer(s) over %d of %d "
                     "steps, %.2f s on %d threads; effective TFLOP/s counts the dense flops "
                     "16*H*B*(I+H)*T' per layer" % (sparsity, layers, Tp, wl.steps, dt, cores),
           "ms_per_layer_step": round(dt / (Tp * layers) * 1e3, 3)}
    oracle.set_threads(1)
    try:
        Tp1, dt1, _ = sized(budget_1core_s)
    finally:
        oracle.set_threads(cores)
    out["single_core"] = {
        "value": round(flops(0, Tp1) / dt1 / 1e12, 6), "unit": "TFLOP/s", "cores": 1,
        "sample": "the same oracle backward of the bottom layer over %d of %d steps, %.2f s on "
                  "one thread" % (Tp1, wl.steps, dt1),
        "ms_per_layer_step": round(dt1 / Tp1 * 1e3, 3)}
    return out


class Runner:
    """Device inputs, forward caches and output buffers of one workload."""

    def __init__(self, L, wl, sparsity, torch):
        from paper_1806_00512_amd.inputs import make_inputs
        self.L, self.wl, self.sparsity, self.torch = L, wl, sparsity, torch
        self.kw = {"P": wl.P, "R": wl.R}  # sparsifying structure of the sparse steps
        dev = torch.device("cuda:0")
        self.st = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
        self.inp = make_inputs(wl, seed=0)
        self.Ws = [torch.from_numpy(w).to(dev).to(self.st) for w in self.inp["Ws"]]
        x0 = torch.from_numpy(self.inp["x"]).to(dev).to(self.st)
        self.dH = torch.from_numpy(self.inp["dH_up"]).to(dev)
        # forward caches (untimed support for the backward pass; the
        # forward is timed on its own by forward_timed)
        self.xs, self.caches, self.houts, self.fws = [], [], [], []
        inp_l = x0
        for li in range(wl.layers):
            I = wl.layer_input(li)
            d = L.dims(wl.steps, wl.batch, I, wl.hidden, self.st)
            self.fws.append(torch.empty(L.fwd_workspace_bytes(d), dtype=torch.uint8, device=dev))
            h_out, cache = L.fwd_cache(inp_l, self.Ws[li], ws=self.fws[li])
            self.xs.append(inp_l)
            self.caches.append(cache)
            self.houts.append(h_out)
            inp_l = h_out
        torch.cuda.synchronize()
        self.sp_bufs = self._buffers(sparsity, dev)
        self.dn_bufs = self._buffers(0.0, dev)
        self.stack_bufs = {}

    def set_structure(self, **kw):
        """Switch the sparse steps to another structure (structure() keywords)."""
        self.kw = kw
        self.sp_bufs = None
        self.stack_bufs = {}
        self.sp_bufs = self._buffers(self.sparsity, self.torch.device("cuda:0"))

    def stack_step(self, sparse):
        """One backward step over all layers as one wavefront stack call
        (lstm_bwd_stack): same results as step(), layers overlapped in time."""
        L, wl = self.L, self.wl
        sp = self.sparsity if sparse else 0.0
        if sparse not in self.stack_bufs:
            o = L.bwd_stack(self.xs, self.Ws, self.caches, self.dH, sparsity=sp, want_dX0=True,
                            **self.kw)
            self.torch.cuda.synchronize()
            ds = [L.dims(wl.steps, wl.batch, wl.layer_input(l), wl.hidden, self.st)
                  for l in range(wl.layers)]
            s = L.structure(**self.kw) if sp > 0 else None
            o["ws"] = self.torch.empty(L.stack_workspace_bytes(ds, sp, s),
                                       dtype=self.torch.uint8, device="cuda:0")
            self.stack_bufs[sparse] = o
        o = self.stack_bufs[sparse]
        L.bwd_stack(self.xs, self.Ws, self.caches, self.dH, sparsity=sp, dXs=o["dX"],
                    dWs=o["dW"], dbs=o["db"], idxs=o["idx"], ws=o["ws"], **self.kw)

    def _buffers(self, sp, dev):
        L, wl, torch = self.L, self.wl, self.torch
        bufs = []
        for li in range(wl.layers):
            I = wl.layer_input(li)
            d = L.dims(wl.steps, wl.batch, I, wl.hidden, self.st)
            s = L.structure(**self.kw) if sp > 0 else None
            ws = torch.empty(L.workspace_bytes(d, sp, s), dtype=torch.uint8, device=dev)
            out = {"dX": torch.empty((wl.steps, I, wl.batch), device=dev),
                   "dW": torch.empty((4 * wl.hidden, I + wl.hidden), device=dev),
                   "db": torch.empty(4 * wl.hidden, device=dev),
                   "dh0": torch.empty((wl.hidden, wl.batch), device=dev),
                   "dc0": torch.empty((wl.hidden, wl.batch), device=dev)}
            if sp > 0:
                ne = L.index_entries(d, sp, s)
                out["idx"] = torch.empty((wl.steps, ne), dtype=torch.int32, device=dev)
            bufs.append((ws, out))
        return bufs

    def step(self, sparse, marks=None):
        """One backward step over all layers (top layer first); marks[li],
        when given, is recorded right after layer li's call."""
        L, wl = self.L, self.wl
        up = self.dH
        for li in reversed(range(wl.layers)):
            if sparse:
                ws, out = self.sp_bufs[li]
                o = L.bwd_structsparse(self.xs[li], self.Ws[li], self.caches[li], up,
                                       sparsity=self.sparsity, out=out, ws=ws, **self.kw)
            else:
                ws, out = self.dn_bufs[li]
                o = L.bwd_dense(self.xs[li], self.Ws[li], self.caches[li], up, out=out, ws=ws)
            if marks is not None:
                marks[li].record()
            up = o["dX"]

    def forward(self, batched=True):
        """Forward pass of every layer (bottom first) into the same caches."""
        for li in range(self.wl.layers):
            self.L.fwd_cache(self.xs[li], self.Ws[li], h_out=self.houts[li],
                             cache=self.caches[li], ws=self.fws[li] if batched else None,
                             batched=batched)

    def forward_timed(self, K, W, batched=True):
        """Mean ms of one forward pass over all layers (HIP events)."""
        torch = self.torch
        for _ in range(W):
            self.forward(batched)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(K):
            self.forward(batched)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K

    def timed(self, schedule, K, W, stack=False):
        """schedule: one cycle of steps (True = sparse); K cycles timed after
        W untimed ones.  Returns mean ms per step, wall ms per step and mean
        ms per layer call (layer times only without stack)."""
        torch, wl = self.torch, self.wl
        for _ in range(W):
            for sp in schedule:
                self.stack_step(sp) if stack else self.step(sp)
        torch.cuda.synchronize()
        if stack:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            w0 = time.perf_counter()
            e0.record()
            for _ in range(K):
                for sp in schedule:
                    self.stack_step(sp)
            e1.record()
            torch.cuda.synchronize()
            n = K * len(schedule)
            return e0.elapsed_time(e1) / n, (time.perf_counter() - w0) / n * 1e3, None

        def ev():
            return torch.cuda.Event(enable_timing=True)

        e0, e1 = ev(), ev()
        spans = []  # (start event, per-layer end events) of every step
        w0 = time.perf_counter()
        e0.record()
        prev = e0
        for _ in range(K):
            for sp in schedule:
                marks = [ev() for _ in range(wl.layers)]
                self.step(sp, marks)
                spans.append((prev, marks))
                prev = marks[0]
        e1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        n = K * len(schedule)
        per_layer = [0.0] * wl.layers
        for start, marks in spans:
            for li in reversed(range(wl.layers)):  # the top layer's call ends first
                per_layer[li] += start.elapsed_time(marks[li])
                start = marks[li]
        return e0.elapsed_time(e1) / n, wall / n * 1e3, [v / n for v in per_layer]


def measure(L, torch, wl, sparsity, steps, warmup, sparse_only=False, kernels=True, fine=None,
            schedules=True, forward=True, mix_cycles_min=1):
    """Backward step timings.  The headline step is the wavefront stack call
    (every layer in one lstm_bwd_stack call); the layers called one after the
    other are timed beside it (with per-layer times).  schedules: the 9 : 1
    (at least mix_cycles_min cycles) and 3 : 1 sparse : dense schedules;
    forward: the forward pass; kernels: the per-kernel timing pass."""
    r = Runner(L, wl, sparsity, torch)
    res = {"runner": r}
    sp_ms, sp_wall, _ = r.timed([True], steps, warmup, stack=True)
    print("%s sparse (stack): %.4f ms/step (wall %.4f)" % (wl.name, sp_ms, sp_wall),
          file=sys.stderr, flush=True)
    res.update(sp_ms=sp_ms, sp_wall=sp_wall)
    if sparse_only:
        return res
    dn_ms, dn_wall, _ = r.timed([False], steps, warmup, stack=True)
    print("%s dense (stack): %.4f ms/step (wall %.4f)" % (wl.name, dn_ms, dn_wall),
          file=sys.stderr, flush=True)
    res.update(dn_ms=dn_ms, dn_wall=dn_wall)
    # the layers one after the other (graph-replayed single-layer calls)
    sq_ms, _, sq_layer = r.timed([True], steps, warmup)
    sqd_ms, _, sqd_layer = r.timed([False], steps, warmup)
    print("%s sequential layers: sparse %.4f, dense %.4f ms/step" % (wl.name, sq_ms, sqd_ms),
          file=sys.stderr, flush=True)
    res.update(sq_ms=sq_ms, sq_layer=sq_layer, sqd_ms=sqd_ms, sqd_layer=sqd_layer)
    if wl.sweep:
        # the workload's sparsity sweep (coarse structure, stack calls)
        pts = []
        for s in wl.sweep:
            if s == 0.0:
                ms = dn_ms
            elif abs(s - sparsity) < 1e-9:
                ms = sp_ms
            else:
                r.sparsity, r.stack_bufs = s, {}
                ms, _, _ = r.timed([True], steps, warmup, stack=True)
            pts.append((s, ms))
            print("%s sweep sparsity %.2f: %.4f ms/step" % (wl.name, s, ms), file=sys.stderr,
                  flush=True)
        r.sparsity, r.stack_bufs = sparsity, {}
        res["sweep"] = pts
    if schedules:
        # the 9 sparse : 1 dense schedule (dense-after-sparse training phases)
        cycles = max(mix_cycles_min, steps // 10)
        mx_ms, _, _ = r.timed([True] * 9 + [False], cycles, 1, stack=True)
        print("%s 9:1 schedule: %.4f ms/step over %d cycles" % (wl.name, mx_ms, cycles),
              file=sys.stderr, flush=True)
        res.update(mix_ms=mx_ms, mix_cycles=cycles)
        # the 3 sparse : 1 dense schedule of dense-after-sparse training
        c3 = max(1, steps // 4)
        m3_ms, _, _ = r.timed([True] * 3 + [False], c3, 1, stack=True)
        print("%s 3:1 schedule: %.4f ms/step" % (wl.name, m3_ms), file=sys.stderr, flush=True)
        res.update(mix3_ms=m3_ms, mix3_cycles=c3)
    if forward:
        # forward pass (batched path, and one pass of the fused per-step path)
        res["fwd_ms"] = r.forward_timed(steps, 1)
        res["fwd_fused_ms"] = r.forward_timed(1, 0, batched=False)
        print("%s forward: %.4f ms (fused per-step kernel %.4f ms)" % (
            wl.name, res["fwd_ms"], res["fwd_fused_ms"]), file=sys.stderr, flush=True)
    if not kernels:
        return res
    # per-kernel HIP-event timing pass (same number of sparse steps, the
    # layers called in turn so that kernels do not overlap); a short spin
    # kernel before and after marks the pass in kernel traces
    torch.cuda.synchronize()
    torch.cuda._sleep(1000)
    L.timing_reset()
    L.timing_enable(True)
    for _ in range(steps):
        r.step(True)
    torch.cuda.synchronize()
    res["kt"] = L.timing_read()
    L.timing_enable(False)
    L.timing_reset()
    torch.cuda._sleep(1000)
    torch.cuda.synchronize()
    for fi, (my, mx) in enumerate(fine or []):
        # fine-grained structure: My x Mx blocks, K = sparsity * nb per slice
        r.set_structure(kind=L.FINE, My=my, Mx=mx)
        fn_ms, fn_wall, _ = r.timed([True], steps, warmup, stack=True)
        print("%s fine (My=%d, Mx=%d): %.4f ms/step" % (wl.name, my, mx, fn_ms), file=sys.stderr,
              flush=True)
        noskip_ms = None
        if my == 32 and mx == 32:
            L.set_option("fine_skip", 0)   # the same call multiplying the removed blocks' zeros
            noskip_ms, _, _ = r.timed([True], steps, warmup, stack=True)
            L.set_option("fine_skip", 1)
            print("%s fine (My=%d, Mx=%d) without skipping: %.4f ms/step" % (wl.name, my, mx,
                                                                           noskip_ms),
                  file=sys.stderr, flush=True)
        L.timing_reset()
        L.timing_enable(True)
        for _ in range(steps):
            r.step(True)
        torch.cuda.synchronize()
        res.setdefault("fine", []).append({"My": my, "Mx": mx, "ms": fn_ms, "noskip_ms": noskip_ms,
                                           "kt": L.timing_read()})
        L.timing_enable(False)
        L.timing_reset()
    return res


def sweep_entries(m):
    """Sparsity sweep points of a measure() result: ms per step of the stack
    call and its speedup over the dense call."""
    return [{"sparsity": s, "ms_per_step": round(ms, 5),
             "speedup_vs_dense": round(m["dn_ms"] / ms, 4)} for s, ms in m["sweep"]]


def measure_training(L, torch, wl, sparsity, steps):
    """Whole training steps (forward, loss gradient, backward of every layer,
    SGD) with the dense-after-sparse trainer: all sparse, all dense, and the
    3 sparse : 1 dense schedule.  Returns mean ms per step of each."""
    from paper_1806_00512_amd.inputs import make_inputs, make_target
    from paper_1806_00512_amd.train import StackConfig, StackTrainer, dense_after_sparse
    dev = torch.device("cuda:0")
    st = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    inp = make_inputs(wl, seed=0)
    cfg = StackConfig(layers=wl.layers, input_size=wl.input_size, hidden=wl.hidden,
                      batch=wl.batch, steps=wl.steps, dtype=st, lr=1e-3, sparsity=sparsity,
                      P=wl.P, R=wl.R)
    tr = StackTrainer(cfg, [torch.from_numpy(w).to(dev).to(st) for w in inp["Ws"]],
                      [torch.from_numpy(b).to(dev) for b in inp["bs"]])
    x = torch.from_numpy(inp["x"]).to(dev).to(st)
    y = torch.from_numpy(make_target(wl)).to(dev)
    del inp
    tr.step(x, y, True)
    tr.step(x, y, False)
    torch.cuda.synchronize()

    def run(schedule):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for sp in schedule:
            tr.step(x, y, sp)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / len(schedule)

    n = max(4, (steps + 3) // 4 * 4)
    res = {"sparse": run([True] * n), "dense": run([False] * n),
           "dense_after_sparse_3to1": run(dense_after_sparse(n, 0.75)), "steps": n}
    print("%s training step: sparse %.3f ms, dense %.3f ms, 3:1 %.3f ms" % (
        wl.name, res["sparse"], res["dense"], res["dense_after_sparse_3to1"]), file=sys.stderr,
        flush=True)
    del tr
    return res


def measure_bidir(L, torch, wl, sparsity, steps):
    """Backward of a bidirectional layer of the workload's bottom-layer shape
    (both directions concurrently in lstm_bwd_bidir) vs the two directions'
    calls one after the other; sparse and dense.  Mean ms per layer call."""
    from paper_1806_00512_amd.inputs import make_inputs
    dev = torch.device("cuda:0")
    st = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    inp = make_inputs(wl, seed=0)
    x = torch.from_numpy(inp["x"]).to(dev).to(st)
    W0 = torch.from_numpy(inp["Ws"][0]).to(dev).to(st)
    Wr = torch.flip(W0, dims=[1]).contiguous()   # a second weight matrix of the same shape
    del inp
    x_rev = L.time_reverse(x)
    _, cf = L.fwd_cache(x, W0)
    _, cr = L.fwd_cache(x_rev, Wr)
    g = torch.Generator(device="cpu").manual_seed(2)
    dH = (torch.randn((wl.steps, 2 * wl.hidden, wl.batch), generator=g) * wl.up_std).to(dev)
    dHf = dH[:, :wl.hidden].contiguous()
    dHr = torch.flip(dH[:, wl.hidden:], dims=[0]).contiguous()
    res = {}

    def tm(f, K):
        f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(K):
            f()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K

    for name, sp in (("sparse", sparsity), ("dense", 0.0)):
        o = L.bwd_bidir(x, x_rev, W0, Wr, cf, cr, dH, sparsity=sp, P=wl.P, R=wl.R)
        d = L.dims(wl.steps, wl.batch, wl.input_size, wl.hidden, st)
        s = L.structure(wl.P, wl.R) if sp > 0 else None
        import ctypes
        n = L.load().lstmss_bidir_workspace_bytes(ctypes.byref(d), float(sp),
                                                  ctypes.byref(s) if s is not None else None)
        ws = torch.empty(int(n), dtype=torch.uint8, device=dev)
        res[name] = tm(lambda: L.bwd_bidir(x, x_rev, W0, Wr, cf, cr, dH, sparsity=sp, P=wl.P,
                                           R=wl.R, out=o, ws=ws), steps)
        outs = []
        for xx, W, cc, up in ((x, W0, cf, dHf), (x_rev, Wr, cr, dHr)):
            wsd = torch.empty(L.workspace_bytes(d, sp, s), dtype=torch.uint8, device=dev)
            od = (L.bwd_structsparse(xx, W, cc, up, sparsity=sp, P=wl.P, R=wl.R, ws=wsd)
                  if sp > 0 else L.bwd_dense(xx, W, cc, up, ws=wsd))
            outs.append((xx, W, cc, up, wsd, od))

        def seq():
            for xx, W, cc, up, wsd, od in outs:
                if sp > 0:
                    L.bwd_structsparse(xx, W, cc, up, sparsity=sp, P=wl.P, R=wl.R, ws=wsd, out=od)
                else:
                    L.bwd_dense(xx, W, cc, up, ws=wsd, out=od)
        res[name + "_directions_in_turn"] = tm(seq, steps)
    print("%s bidirectional bottom layer: sparse %.3f ms (directions in turn %.3f), dense %.3f "
          "(%.3f)" % (wl.name, res["sparse"], res["sparse_directions_in_turn"], res["dense"],
                      res["dense_directions_in_turn"]), file=sys.stderr, flush=True)
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: the library runs on one GPU (--gpus 1); sharding across GPUs is "
              "not implemented", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_1806_00512_amd.lstmss as L
    from paper_1806_00512_amd.inputs import WORKLOADS

    L.load()
    if args.serial:
        L.set_option("side_stream", 0)
    wl = WORKLOADS[args.workload]
    sparsity = wl.sparsity if args.sparsity is None else args.sparsity
    st = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    es = 2 if wl.dtype == "bf16" else 4

    if args.calibration_copy_mib > 0:
        n = args.calibration_copy_mib * (1 << 20) // 4
        a = torch.ones(n, device="cuda:0")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        print("calibration copy: %d MiB read, %d MiB written" % (args.calibration_copy_mib,
                                                                  args.calibration_copy_mib),
              file=sys.stderr, flush=True)
        del a, b

    fine = None if args.no_fine else (args.fine_my, args.fine_mx)
    if fine is not None:
        # the paper's blocks, and blocks shaped like the 32 x 32 MFMA operand
        # blocks (their products skip the removed blocks)
        cand = [fine] + ([(32, 32)] if tuple(fine) != (32, 32) else [])
        fine = []
        for my, mx in cand:
            nb = -(-wl.batch // my)
            if abs(sparsity * nb - round(sparsity * nb)) > 1e-6 * nb or (4 * wl.hidden) % mx:
                print("fine structure My=%d, Mx=%d skipped: sparsity %g of %d blocks per slice "
                      "is not a whole number of blocks, or Mx does not divide 4H"
                      % (my, mx, sparsity, nb), file=sys.stderr, flush=True)
                continue
            fine.append((my, mx))
    m = measure(L, torch, wl, sparsity, args.steps, args.warmup, args.sparse_only, fine=fine,
                mix_cycles_min=2)
    if args.sparse_only:
        return
    sp_ms, dn_ms, kt = m["sp_ms"], m["dn_ms"], m["kt"]

    def flops_of(w, frac_kept=None):
        tot = 0.0
        for l in range(w.layers):
            f = 16.0 * w.hidden * w.batch * (w.layer_input(l) + w.hidden) * w.steps
            tot += f if frac_kept is None else f * frac_kept[l]
        return tot

    dense_flops = flops_of(wl)
    roofs, sp_kps = roofline_all(L, wl, sparsity, kt, args.steps)
    exec_flops = flops_of(wl, [k / (4 * wl.hidden) for k in sp_kps])
    kernels = kernel_table(kt, args.steps)
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
                   "S": int(round(sparsity * wl.R)), "storage": wl.dtype,
                   "side_stream": "off" if args.serial else "auto",
                   "schedule": "wavefront stack call (lstm_bwd_stack)"},
        "dense_ms_per_step": round(dn_ms, 5),
        "speedup_vs_dense": round(dn_ms / sp_ms, 4),
        "algorithmic_tflops": round(exec_flops / (sp_ms / 1e3) / 1e12, 4),
        "dense_tflops": round(dense_flops / (dn_ms / 1e3) / 1e12, 4),
        "sequential_layers": {
            "note": "the layers' backward calls one after the other (each replayed from its "
                    "HIP graph) instead of one wavefront stack call",
            "ms_per_step": round(m["sq_ms"], 5), "dense_ms_per_step": round(m["sqd_ms"], 5),
            "speedup_vs_dense": round(m["sqd_ms"] / m["sq_ms"], 4),
            "per_layer_ms": {"sparse": [round(v, 5) for v in m["sq_layer"]],
                             "dense": [round(v, 5) for v in m["sqd_layer"]]}},
        "mixed_9sparse_1dense": {"ms_per_step": round(m["mix_ms"], 5), "cycles": m["mix_cycles"],
                                 "formula_ms": round((9 * sp_ms + dn_ms) / 10, 5),
                                 "speedup_vs_dense": round(dn_ms / m["mix_ms"], 4)},
        "mixed_3sparse_1dense": {"ms_per_step": round(m["mix3_ms"], 5),
                                 "cycles": m["mix3_cycles"],
                                 "speedup_vs_dense": round(dn_ms / m["mix3_ms"], 4)},
        "wall_ms_per_step": {"sparse": round(m["sp_wall"], 5), "dense": round(m["dn_wall"], 5)},
        "kernels": kernels,
        "roofline": roofs[dominant],
        "roofline_all": roofs,
    }
    fwd_flops = sum(8.0 * wl.hidden * wl.batch * (wl.layer_input(l) + wl.hidden) * wl.steps
                    for l in range(wl.layers))
    result["forward"] = {"ms_per_step": round(m["fwd_ms"], 5),
                         "tflops": round(fwd_flops / (m["fwd_ms"] / 1e3) / 1e12, 4),
                         "fused_per_step_kernel_ms": round(m["fwd_fused_ms"], 5),
                         "note": "forward of every layer over all steps (fills the backward "
                                 "cache); flops 8*H*B*(I+H)*T per layer"}
    if not args.no_train:
        tm = measure_training(L, torch, wl, sparsity, args.steps)
        result["training"] = {
            "ms_per_step": {k: round(tm[k], 5) for k in ("sparse", "dense",
                                                          "dense_after_sparse_3to1")},
            "speedup_vs_dense": {"sparse": round(tm["dense"] / tm["sparse"], 4),
                                 "dense_after_sparse_3to1":
                                     round(tm["dense"] / tm["dense_after_sparse_3to1"], 4)},
            "steps_timed": tm["steps"],
            "note": "whole training step: forward of every layer, loss gradient, backward of "
                    "every layer (no input gradient for the bottom layer), SGD; synthetic "
                    "regression target"}
    if not args.no_bidir:
        bd = measure_bidir(L, torch, wl, sparsity, args.steps)
        result["bidirectional"] = {
            "ms_per_layer_call": {k: round(v, 5) for k, v in bd.items()},
            "speedup_vs_dense": round(bd["dense"] / bd["sparse"], 4),
            "note": "backward of one bidirectional layer of the bottom layer's shape (both "
                    "directions concurrently, lstm_bwd_bidir) vs the two directions' calls in "
                    "turn"}
    for fm in m.get("fine", []):
        nb = -(-wl.batch // fm["My"])
        fk = kernel_table(fm["kt"], args.steps)
        entry = {"My": fm["My"], "Mx": fm["Mx"], "blocks_per_slice": nb,
                 "K": int(round(sparsity * nb)), "ms_per_step": round(fm["ms"], 5),
                 "speedup_vs_dense": round(dn_ms / fm["ms"], 4),
                 "value": round(dense_flops / (fm["ms"] / 1e3) / 1e12, 4), "unit": "TFLOP/s",
                 "kernels": fk}
        if fm["noskip_ms"] is not None:
            entry["without_skipping_ms_per_step"] = round(fm["noskip_ms"], 5)
        if (fm["My"], fm["Mx"]) == (32, 32):
            entry["note"] = ("blocks shaped like the 32 x 32 MFMA operand blocks: the products "
                             "skip the removed blocks")
            result["fine_mfma_blocks"] = entry
        else:
            result["fine"] = entry
    if "sweep" in m:
        result["sparsity_sweep"] = sweep_entries(m)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, m["runner"].inp, sparsity)
    del m
    if not args.no_also:
        also = []
        for name in ALSO_WORKLOADS:
            if name == wl.name:
                continue
            w2 = WORKLOADS[name]
            k2 = max(args.steps, 10)
            mixed = w2.dtype == "bf16"   # the bf16 workload is the 9 : 1 schedule's
            m2 = measure(L, torch, w2, w2.sparsity, k2, args.warmup, schedules=mixed,
                         forward=False, mix_cycles_min=2)
            r2, _ = roofline_all(L, w2, w2.sparsity, m2["kt"], k2)
            e2 = {"workload": name, "dtype": w2.dtype,
                  "config": {"layers": w2.layers, "input_size": w2.input_size,
                             "hidden": w2.hidden, "batch": w2.batch, "seq_len": w2.steps,
                             "sparsity": w2.sparsity, "P": w2.P, "R": w2.R},
                  "ms_per_step": round(m2["sp_ms"], 5),
                  "dense_ms_per_step": round(m2["dn_ms"], 5),
                  "speedup_vs_dense": round(m2["dn_ms"] / m2["sp_ms"], 4),
                  "sequential_layers_ms_per_step": {"sparse": round(m2["sq_ms"], 5),
                                                    "dense": round(m2["sqd_ms"], 5)},
                  "value": round(flops_of(w2) / (m2["sp_ms"] / 1e3) / 1e12, 4),
                  "unit": "TFLOP/s",
                  "kernels": kernel_table(m2["kt"], k2),
                  "roofline": r2[max(r2, key=lambda k: m2["kt"][k][0])],
                  "roofline_all": r2}
            if mixed:
                e2["mixed_9sparse_1dense"] = {
                    "ms_per_step": round(m2["mix_ms"], 5), "cycles": m2["mix_cycles"],
                    "formula_ms": round((9 * m2["sp_ms"] + m2["dn_ms"]) / 10, 5),
                    "speedup_vs_dense": round(m2["dn_ms"] / m2["mix_ms"], 4)}
                e2["mixed_3sparse_1dense"] = {
                    "ms_per_step": round(m2["mix3_ms"], 5), "cycles": m2["mix3_cycles"],
                    "speedup_vs_dense": round(m2["dn_ms"] / m2["mix3_ms"], 4)}
            if "sweep" in m2:
                e2["sparsity_sweep"] = sweep_entries(m2)
            also.append(e2)
            del m2
            torch.cuda.empty_cache()
        result["also"] = also
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
