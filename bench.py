#!/usr/bin/env python3
"""Benchmark of the kernel-quantization hot path on one MI355X.

Workload (one step): the ResNet-18-shaped stack of 3x3 convolutions (16 layers,
1,220,608 kernels, synthetic Laplace weights), one codebook of k = 256 entries per
layer started from k distinct kernels (kq_forgy_select), then, in one library call
(kq_compress_stack):
  * 30 Lloyd rounds (assign + update) and a final assignment on every layer,
  * the final member counts,
  * 6-bit weighted k-means quantization of every codebook (Sec. 3.2),
  * packing of the 8-bit indices and of the 6-bit codes (Eq. 4),
  * reconstruction of every weight tensor from the packed indices and the
    dequantised codebook, and its squared error against the original weights.

value = kernels x Lloyd rounds / step time (everything above inside the step; inputs
resident in HBM before the timed region).  The dominant kernel, the assignment, is
timed inside the timed steps: each step has the library record a pair of HIP events
around one round's assignment launch (round s mod 30 in step s), and the mean of those
launches prices it against the FP32 peak.  A diagnostic line on stderr adds the other
launches (warm and after a 1 GiB cache flush), the per-layer report of Sec. 4.2.1
(l2 error, Eq. 4, 6, 7 for K and K+C) and the codebook-retraining step of Eq. (2).
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "kernels assigned/sec per Lloyd iter (ResNet-18 stack, K=256); % FP32 peak; HBM GB/s"
FP32_PEAK_TFLOPS = 157.3     # MI355X dense FP32 (matrix cores and vector)
HBM_PEAK_GBS = 8000.0
FLUSH_BYTES = 1 << 30        # a cold measurement writes this much, then reads as much of another buffer


# workloads: layer generator, codebook size, Lloyd rounds, first seed of the initial codebooks, description
CONFIGS = {
    "resnet18": ("resnet18_stack", 256, 30, 2000, "resnet18-3x3-stack (16 layers, 1,220,608 kernels, Laplace)"),
    "vgg16": ("vgg16_stack", 256, 30, 1000,
              "vgg16-3x3-stack (13 layers, 1,634,496 kernels, normal; conv1 k clamped to 192)"),
    "single": ("single_layer", 256, 20, 1, "single 64x64 layer (4096 kernels, normal)"),
    "stress": ("stress_layer", 4096, 10, 4000, "stress 1024x1024 layer (1,048,576 kernels from 4096 clusters)"),
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="resnet18", choices=sorted(CONFIGS),
                    help="workload (default: the ResNet-18-shaped stack, the headline metric)")
    ap.add_argument("--iters", type=int, default=None, help="Lloyd rounds per layer (default: the config's)")
    ap.add_argument("--k", type=int, default=None, help="codebook size (default: the config's)")
    ap.add_argument("--yinyang", action="store_true",
                    help="run each layer's Lloyd rounds with Yinyang assignments (Sec. 4.1; the same result)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-diag", action="store_true", help="skip the diagnostic line")
    ap.add_argument("--cpu-iters", type=int, default=2, help="Lloyd rounds of the oracle sample")
    ap.add_argument("--row", choices=["lloyd", "fc", "search", "report"], default="lloyd",
                    help="lloyd: the step above (default); fc: the fully-connected-layer quantizer "
                         "(kq_quantize_scalars, 6 bits, 30 rounds) on the VGG-16 fc6/fc7/fc8 shapes; "
                         "search: the codebook-size search (kq_search_codebook_size) on the "
                         "ResNet-18 conv1 shape; report: only the per-layer compression report")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="after the timed steps, copy MIB MiB device to device three times (a plain copy "
                         "kernel of known size, the scale for hardware byte counters)")
    return ap.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "assign_traffic.json")
TRAFFIC_SOURCES = ["paper_2003_05148_amd/csrc/kq_assign.hip", "paper_2003_05148_amd/csrc/kq_internal.h"]


def assign_traffic():
    """HBM bytes per launch of the assignment kernel from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, scaled by the same counters on a plain copy), or None when
    the kernel's sources have changed since the counters were taken."""
    import hashlib
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    if rec.get("sources_sha256") != h.hexdigest():
        return None
    return rec["bytes_per_launch"]


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def host_cores() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    env = os.environ.get("OMP_NUM_THREADS")
    return max(1, min(n, int(env))) if env and env.isdigit() else n


def cpu_baseline(layers, C0, iters, budget=1e9):
    """The CPU oracle (plain C) on a bounded sample: `iters` Lloyd rounds plus the final
    assignment on every layer, each layer cut to its first rows when the full stack would
    exceed `budget` (kernel x entry x round) units; once on one thread, once with the
    assignment loop on all host cores (same results)."""
    import oracle
    work = sum(L.n * L.k * (iters + 1) for L in layers)
    f = min(1.0, budget / work)

    def run(threads):
        oracle.set_threads(threads)
        t0 = time.perf_counter()
        n = 0
        for L, c in zip(layers, C0):
            m = min(L.n, max(L.k, int(L.n * f)))
            oracle.fit(L.X[:m], c, iters)
            n += m
        return n, time.perf_counter() - t0

    n, dt1 = run(1)
    cores = host_cores()
    _, dtn = run(cores)
    oracle.set_threads(1)
    rows = "all rows" if f >= 1.0 else f"the first {100 * f:.1f} % of the rows"
    return {"value": n * iters / dtn, "unit": "kernels/s", "cores": cores, "kind": "oracle",
            "single_thread_value": n * iters / dt1, "cpu_model": cpu_model(),
            "sample": f"{iters} Lloyd rounds + final assignment on {rows} of all {len(layers)} layers "
                      f"({n} kernels, k={layers[0].k}): {dtn:.1f} s with the assignment loop on {cores} "
                      f"threads, {dt1:.1f} s on one"}


def bench_fc(args, kq, torch):
    """kq_quantize_scalars on N(0, 2/fan_in) weights of the VGG-16 fully-connected shapes."""
    import math
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(6)
    stream = torch.cuda.current_stream(dev)
    rows = []
    for name, (o, i) in [("fc6", (4096, 25088)), ("fc7", (4096, 4096)), ("fc8", (1000, 4096))]:
        m = o * i
        v = torch.randn(m, device=dev, generator=g) * math.sqrt(2.0 / i)
        out = kq.kq_quantize_scalars(v, 6, 30)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            out = kq.kq_quantize_scalars(v, 6, 30)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        r = int(out[3].item())
        rows.append({"layer": name, "scalars": m, "rounds": r, "ms": ms, "us_per_pass": 1e3 * ms / (r + 1),
                     "GBps_at_5B_per_scalar_pass": 5.0 * m * (r + 1) / (ms * 1e-3) / 1e9})
    tot_ms = sum(r_["ms"] for r_ in rows)
    print(json.dumps({"metric": "FC-layer 6-bit scalar quantization: scalars per second (30 rounds)",
                      "value": sum(r_["scalars"] for r_ in rows) / (tot_ms * 1e-3), "unit": "scalars/s",
                      "n_gpus": 1, "steps": args.steps, "dtype": "f32", "data": "synthetic",
                      "config": {"workload": "VGG-16 fc6 25088x4096, fc7 4096x4096, fc8 4096x1000, N(0, 2/fan_in)"},
                      "rows": rows}))


def bench_search(args, kq, torch, synth):
    """kq_search_codebook_size on the ResNet-18 conv1 shape (alpha = 0.3, r = 0.5, 8
    iterations, 30 Lloyd rounds per fit)."""
    dev = torch.device("cuda:0")
    L = synth.resnet18_stack(k=256, layers=1)[0]
    n_init = int(0.3 * L.n)
    cand = L.X[kq.kq_forgy_select(L.X, n_init, 7)]
    Xd, Cd = torch.from_numpy(L.X).to(dev), torch.from_numpy(cand).to(dev)
    kq.kq_search_codebook_size(Xd, Cd, 0.5, 8, 30)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        k, C, idx, trials, d0 = kq.kq_search_codebook_size(Xd, Cd, 0.5, 8, 30)
    torch.cuda.synchronize()
    ms = 1e3 * (time.perf_counter() - t0) / args.steps
    print(json.dumps({"metric": "codebook-size search: fits per second (30 Lloyd rounds each)",
                      "value": (len(trials) + 1) / (ms * 1e-3), "unit": "fits/s", "n_gpus": 1,
                      "steps": args.steps, "dtype": "f32", "data": "synthetic",
                      "config": {"workload": f"resnet18 conv1 64x64 ({L.n} kernels), n_init {n_init}, "
                                             "r = 0.5, 8 iterations"},
                      "ms_per_search": ms, "k": int(k), "trials": [int(t[0]) for t in trials]}))


def layer_report(kq, torch, layers, comp, T):
    """Sec. 4.2.1 per layer: the l2 reconstruction error (mean squared error per weight) of
    K (the fp32 codebook: the final distortion / 9n) and of K+C (6-bit codebook, weighted
    k-means as in Sec. 3.2, and the uniform grid), and Eq. (4), (6), (7) for K and K+C."""
    dev = comp.device
    uni = kq.kq_quantize_codebook_stack(comp.C, comp.counts, 6, kq.KQ_CBQ_UNIFORM, 0)
    sq_uni = torch.zeros(len(layers), dtype=torch.float64, device=dev)
    recon = [{"idx": comp.idx[i], "n": L.n, "C": uni[i][2], "W_ref": comp.X[i], "sq_error": sq_uni[i:i + 1]}
             for i, L in enumerate(layers)]
    kq.kq_reconstruct_stack(recon)
    torch.cuda.synchronize()
    sq_w, sq_u = comp.sq_error.cpu().tolist(), sq_uni.cpu().tolist()
    rows = []
    for i, L in enumerate(layers):
        p = 9 * L.n
        B_k, cr_k, beta_k = kq.kq_accounting(L.n, L.k, 32)
        B_kc, cr_kc, beta_kc = kq.kq_accounting(L.n, L.k, 6)
        rows.append({"layer": L.name, "n": L.n, "k": L.k, "index_bits": kq.index_bits(L.k),
                     "mse_K": float(comp.distortion[i][T].item()) / p, "mse_KC_wkmeans": sq_w[i] / p,
                     "mse_KC_uniform": sq_u[i] / p, "B_K": B_k, "CR_K": cr_k, "beta_K": beta_k,
                     "B_KC": B_kc, "CR_KC": cr_kc, "beta_KC": beta_kc})
    n_tot = sum(L.n for L in layers)
    tot = {"beta_K": sum(r["B_K"] for r in rows) / (9 * n_tot), "beta_KC": sum(r["B_KC"] for r in rows) / (9 * n_tot)}
    tot["CR_K"], tot["CR_KC"] = 32 / tot["beta_K"], 32 / tot["beta_KC"]
    return rows, tot


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the path is measured "
              "on a single MI355X and is not sharded across GPUs.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2003_05148_amd as kq
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.row == "fc":
        return bench_fc(args, kq, torch)
    if args.row == "search":
        return bench_search(args, kq, torch, synth)
    gen, k_default, iters_default, seed0, desc = CONFIGS[args.config]
    k = args.k if args.k is not None else k_default
    T = args.iters if args.iters is not None else iters_default
    layers = getattr(synth, gen)(k=k)            # kernels and codebook sizes (k clamped to the distinct kernels)
    n_total = sum(L.n for L in layers)
    C0 = [np.ascontiguousarray(L.X[kq.kq_forgy_select(L.X, L.k, seed0 + i)]) for i, L in enumerate(layers)]

    # inputs resident in HBM before timing
    X = [torch.from_numpy(L.X).to(dev) for L in layers]
    C0d = [torch.from_numpy(c).to(dev) for c in C0]
    comp = kq.Compression(X, C0d, iters=T, bits=6, mode=kq.KQ_CBQ_WKMEANS, cbq_iters=30)
    stream = torch.cuda.current_stream(dev)

    if args.yinyang:
        return bench_yinyang(args, kq, torch, layers, X, C0d, comp, T, desc, k)

    # one event pair per timed step, recorded by the library around one round's assignment
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for a, b in ev:                              # torch creates its events on their first record
        a.record(stream)
        b.record(stream)
    for _ in range(args.warmup):
        comp.run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        comp.run(round_events={s % T: ev[s]} if T > 0 else None)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = 1e3 * elapsed / args.steps
    assign_ms = float(np.mean([a.elapsed_time(b) for a, b in ev])) if T > 0 else 0.0
    flops = 18.0 * sum(L.k * L.n for L in layers)   # 9 multiply-adds per (kernel, entry) pair
    achieved = flops / (assign_ms * 1e-3) / 1e12 if assign_ms > 0 else 0.0
    fused = max(L.k for L in layers) <= 256

    if args.copy_probe > 0:
        src = torch.ones(args.copy_probe << 18, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    if args.row == "report":
        rows, tot = layer_report(kq, torch, layers, comp, T)
        print(json.dumps({"report": rows, "stack": tot, "config": desc, "k": k, "lloyd_rounds": T}))
        return
    if not args.no_diag:
        print(json.dumps({"diag": diagnostics(kq, torch, np, layers, comp, T, fused, stream)}), file=sys.stderr,
              flush=True)

    result = {
        "metric": METRIC,
        "value": n_total * T / (ms_step * 1e-3),
        "unit": "kernels/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{desc} k={k}: {T} Lloyd rounds + final assignment, "
                               "6-bit weighted codebook quantization, index/code packing, packed reconstruction "
                               "(one kq_compress_stack call per step)",
                   "layers": len(layers), "kernels": n_total, "k": k, "lloyd_rounds": T, "codebook_bits": 6},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / FP32_PEAK_TFLOPS,
                     "traffic": assign_traffic() if (args.config, k) == ("resnet18", 256) else None,
                     "kernel": ("assign_kernel<2, true> (member sums fused)" if fused else "assign_kernel<2, false>")
                               + f": one Lloyd round's launch per timed step (rounds 0..{min(args.steps, T) - 1}), "
                                 "whole stack per launch",
                     "pricing": "bf16-split MFMA screening + exact fp32 rescoring; the method's fp32 flops "
                                "(18 k per kernel) priced at the 157.3 TFLOP/s FP32 peak"},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(layers, C0, args.cpu_iters)
    print(json.dumps(result), flush=True)


def head_start(torch, stream, ms=2.0):
    """Queue about `ms` of GPU spinning (no memory traffic) so that the launches queued
    after it are timed by the GPU's progress, not by how fast the host enqueues them."""
    if not hasattr(head_start, "cycles_per_ms"):   # calibrate the spin once, on a long spin
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        torch.cuda._sleep(5_000_000)
        b.record(stream)
        torch.cuda.synchronize()
        head_start.cycles_per_ms = 5_000_000 / max(a.elapsed_time(b), 1e-3)
    torch.cuda._sleep(int(head_start.cycles_per_ms * ms))


class LaunchTimer:
    """Median duration (ms) of a call's launches between two HIP events, over `reps`
    calls queued behind a head start; `prep` runs (untimed) before each call; with the
    flush buffers, 1 GiB is written and another 1 GiB read before each call, so that it
    starts from caches that hold none of its data and nothing dirty.  The events are
    created once and reused."""

    def __init__(self, torch, stream, reps=5):
        self.torch, self.stream = torch, stream
        self.ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in self.ev:
            a.record(stream)
            b.record(stream)
        torch.cuda.synchronize()

    def __call__(self, fn, prep=None, flush=None):
        import statistics
        head_start(self.torch, self.stream)
        for a, b in self.ev:
            if prep:
                prep()
            if flush is not None:      # 1 GiB written, then 1 GiB of another buffer read: the caches
                flush[0].zero_()         # end up holding clean lines of the second buffer only
                flush[1].sum()
            a.record(self.stream)
            fn()
            b.record(self.stream)
        self.torch.cuda.synchronize()
        return statistics.median(a.elapsed_time(b) for a, b in self.ev)


def diagnostics(kq, torch, np, layers, comp, T, fused, stream):
    """Per-launch times of the other steps, through the per-step stack calls on the state
    the timed steps left (the same kernels and launch configurations), warm and after a
    1 GiB flush; the per-layer report; the Eq. (2) codebook step."""
    dev = comp.device
    n_total = sum(L.n for L in layers)
    flush = (torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev),
             torch.zeros(FLUSH_BYTES, dtype=torch.uint8, device=dev))
    st = kq.Stack(comp.X, [c.clone() for c in comp.C], iters=1)
    reps = 5

    timer = LaunchTimer(torch, stream, reps)

    def both(fn, prep=None):
        if prep:
            prep()
        fn()                                       # caches warm
        return timer(fn, prep), timer(fn, prep, flush)

    d = {}
    # the shifts of the layers' sums once (an update that finds them), then each step's launches alone
    kq.kq_update_stack(st)
    if fused:
        d["assign_fused_ms"] = both(lambda: kq.kq_assign_stack(st, distortion=False, fused_sums=True,
                                                               reuse_shifts=True))
        d["finish_ms"] = both(lambda: kq.kq_update_stack(st, distortion_from_assign=True, sums_from_assign=True),
                              prep=lambda: kq.kq_assign_stack(st, distortion=False, fused_sums=True,
                                                              reuse_shifts=True))
    d["assign_plain_ms"] = both(lambda: kq.kq_assign_stack(st, distortion=False))
    upd = both(lambda: kq.kq_update_stack(st, reuse_shifts=True))
    d["update_separate_ms"] = upd                              # update_kernel + finish, 40 B per kernel read
    d["update_separate_GBps"] = [40.0 * n_total / (t * 1e-3) / 1e9 for t in upd]
    # outputs made once: the timed calls enqueue the launch only
    cbq_out = kq.kq_quantize_codebook_stack(comp.C, comp.counts, 6, kq.KQ_CBQ_WKMEANS, 30)
    d["cbq_wkmeans_ms"] = both(lambda: kq.kq_quantize_codebook_stack(comp.C, comp.counts, 6, kq.KQ_CBQ_WKMEANS, 30,
                                                                     out=cbq_out))
    jobs = [(comp.idx[i], comp.index_bits[i], comp.packed_idx[i]) for i in range(len(layers))] + \
           [(comp.codes[i], 6, comp.packed_codes[i]) for i in range(len(layers))]
    d["pack_ms"] = both(lambda: kq.kq_pack_bits_stack(jobs))
    rec_err = [{"packed": comp.packed_idx[i], "bits": comp.index_bits[i], "n": L.n, "C": comp.C_hat[i],
                "W_hat": comp.W_hat[i], "W_ref": comp.X[i], "sq_error": comp.sq_error[i:i + 1]}
               for i, L in enumerate(layers)]
    rec_plain = [{"idx": comp.idx[i], "n": L.n, "C": comp.C_hat[i], "W_hat": comp.W_hat[i]}
                 for i, L in enumerate(layers)]
    ws = torch.zeros(max(256, kq.recon_workspace_bytes(rec_err)), dtype=torch.uint8, device=dev)
    d["reconstruct_packed_with_error_ms"] = both(lambda: kq.kq_reconstruct_stack(rec_err, workspace=ws))
    rp = both(lambda: kq.kq_reconstruct_stack(rec_plain, workspace=ws))
    d["reconstruct_plain_ms"] = rp                             # 4 B index read + 36 B row written per kernel
    d["reconstruct_plain_GBps"] = [40.0 * n_total / (t * 1e-3) / 1e9 for t in rp]
    d["warm_cold_note"] = ("each pair [warm, cold] in ms: median of 5 calls queued behind a head start, then of "
                           "5 calls each after writing 1 GiB and reading another 1 GiB (events around the call)")
    # Eq. (2) codebook retraining step on the same stack: synthetic gradients of the kernels'
    # shape and the final assignment, one launch set per step
    gst = kq.Stack([x * 1e-3 for x in comp.X], [c.clone() for c in comp.C])
    for i in range(len(layers)):
        gst.idx[i].copy_(comp.idx[i])
    g = both(lambda: kq.kq_codebook_grad_step_stack(gst, 0.01))
    d["grad_step_ms"] = g
    d["grad_step_GBps"] = [40.0 * n_total / (t * 1e-3) / 1e9 for t in g]
    rows, tot = layer_report(kq, torch, layers, comp, T)
    d["report"] = rows
    d["report_stack"] = tot
    del flush
    return d


def bench_yinyang(args, kq, torch, layers, X, C0d, comp, T, desc, k):
    """Each layer's fit with Yinyang assignments (Sec. 4.1): the same result as the Lloyd
    path; the distances its bounds leave to evaluate, over its whole time."""
    import numpy as np
    dev = comp.device
    stream = torch.cuda.current_stream(dev)
    yy_ws = [torch.empty(kq.lib.kq_yinyang_workspace_bytes(L.n, L.k, 0), dtype=torch.uint8, device=dev)
             for L in layers]
    stats = [torch.zeros(max(T, 1), 3, dtype=torch.int64, device=dev) for _ in layers]

    def step():
        for i in range(len(layers)):
            kq.kq_fit_layer_yinyang(X[i], C0d[i], T, C=comp.C[i], idx=comp.idx[i], counts=comp.counts[i],
                                    distortion=comp.distortion[i], stats=stats[i], workspace=yy_ws[i])
        kq.kq_quantize_codebook_stack(comp.C, comp.counts, 6, kq.KQ_CBQ_WKMEANS, 30)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms_step = 1e3 * (time.perf_counter() - t0) / args.steps
    st = [s.cpu().numpy() for s in stats]
    evals = sum(L.n * L.k + int(s[:T, 2].sum()) for L, s in zip(layers, st))
    full = sum(L.n * L.k * (T + 1) for L in layers)
    achieved = 18.0 * evals / (ms_step * 1e-3) / 1e12
    n_total = sum(L.n for L in layers)
    print(json.dumps({"metric": METRIC, "value": n_total * T / (ms_step * 1e-3), "unit": "kernels/s", "n_gpus": 1,
                      "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
                      "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
                      "config": {"workload": f"{desc} k={k}: {T} Yinyang Lloyd rounds + final assignment per layer, "
                                             "6-bit weighted codebook quantization", "assignment": "yinyang"},
                      "roofline": {"bound": "alu", "achieved": achieved, "peak": FP32_PEAK_TFLOPS / 2,
                                   "unit": "TFLOP/s", "frac": achieved / (FP32_PEAK_TFLOPS / 2), "traffic": None,
                                   "kernel": "kq_fit_layer_yinyang (all launches of the fits, whole step)"},
                      "yinyang": {"distance_evaluations": evals, "lloyd_equivalent": full,
                                  "evaluated_fraction": evals / full}}), flush=True)


if __name__ == "__main__":
    main()
