#!/usr/bin/env python3
"""Benchmark of the kernel-quantization hot path on one MI355X.

Workload (one step): the ResNet-18-shaped stack of 3x3 convolutions (16 layers,
1,220,608 kernels, synthetic Laplace weights), one codebook of k = 256 entries per
layer, then
  * 30 Lloyd rounds (assign + update) and a final assignment on every layer,
  * the final member counts,
  * 6-bit weighted k-means quantization of every codebook (Sec. 3.2),
  * packing of the 8-bit indices and of the 6-bit codes (Eq. 4),
  * reconstruction of every weight tensor from the packed indices and the
    dequantised codebook, and its squared error against the original weights.

value = kernels x Lloyd rounds / step time (everything above inside the step).
The assignment kernel's own duration is measured with HIP events on the stream it
runs on, in one instrumented step after the timed ones, and priced against the FP32
peak.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "kernels assigned/sec per Lloyd iter (ResNet-18 stack, K=256); % FP32 peak; HBM GB/s"
FP32_PEAK_TFLOPS = 157.3     # MI355X dense FP32 (matrix cores and vector)
HBM_PEAK_GBS = 8000.0


# workloads: layer generator, codebook size, Lloyd rounds, description
CONFIGS = {
    "resnet18": ("resnet18_stack", 256, 30, "resnet18-3x3-stack (16 layers, 1,220,608 kernels, Laplace)"),
    "vgg16": ("vgg16_stack", 256, 30, "vgg16-3x3-stack (13 layers, 1,634,496 kernels, normal; conv1 k clamped to 192)"),
    "single": ("single_layer", 256, 20, "single 64x64 layer (4096 kernels, normal)"),
    "stress": ("stress_layer", 4096, 10, "stress 1024x1024 layer (1,048,576 kernels from 4096 clusters)"),
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="resnet18", choices=sorted(CONFIGS),
                    help="workload (default: the ResNet-18-shaped stack, the headline metric)")
    ap.add_argument("--iters", type=int, default=None, help="Lloyd rounds per layer (default: the config's)")
    ap.add_argument("--k", type=int, default=None, help="codebook size (default: the config's)")
    ap.add_argument("--yinyang", action="store_true",
                    help="run each layer's Lloyd rounds with Yinyang assignments (Sec. 4.1; the same result)")
    ap.add_argument("--unfused", action="store_true",
                    help="run the update as its own pass over the kernels (the member sums are not fused "
                         "into the assignment)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-iters", type=int, default=2, help="Lloyd rounds of the oracle sample")
    ap.add_argument("--row", choices=["lloyd", "fc", "search"], default="lloyd",
                    help="lloyd: the step above (default); fc: the fully-connected-layer quantizer "
                         "(kq_quantize_scalars, 6 bits, 30 rounds) on the VGG-16 fc6/fc7/fc8 shapes; "
                         "search: the codebook-size search (kq_search_codebook_size) on the "
                         "ResNet-18 conv1 shape")
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


def cpu_baseline(layers, iters, budget=1e9):
    """The CPU oracle (single-threaded plain C) on a bounded sample: `iters` Lloyd
    rounds plus the final assignment on every layer, each layer cut to its first rows
    when the full stack would exceed `budget` (kernel x entry x round) units."""
    import oracle
    work = sum(L.n * L.k * (iters + 1) for L in layers)
    f = min(1.0, budget / work)
    t0 = time.perf_counter()
    n = 0
    for L in layers:
        m = min(L.n, max(L.k, int(L.n * f)))
        oracle.fit(L.X[:m], L.C0, iters)
        n += m
    dt = time.perf_counter() - t0
    rows = "all rows" if f >= 1.0 else f"the first {100 * f:.1f} % of the rows"
    return {"value": n * iters / dt, "unit": "kernels/s", "cores": 1, "kind": "oracle",
            "sample": f"{iters} Lloyd rounds + final assignment on {rows} of all {len(layers)} layers "
                      f"({n} kernels, k={layers[0].k}), {dt:.1f} s"}


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
    cand = L.X[synth.distinct_init(L.X, n_init, 7)]
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
    gen, k_default, iters_default, desc = CONFIGS[args.config]
    k = args.k if args.k is not None else k_default
    T = args.iters if args.iters is not None else iters_default
    layers = getattr(synth, gen)(k=k)
    n_total = sum(L.n for L in layers)

    # inputs resident in HBM before timing
    X = [torch.from_numpy(L.X).to(dev) for L in layers]
    sizes = [L.k * 9 for L in layers]
    C0flat = torch.from_numpy(np.concatenate([L.C0.reshape(-1) for L in layers])).to(dev)
    st = kq.Stack(X, [torch.empty(L.k, 9, device=dev) for L in layers], iters=T)
    # make the stack's codebooks views of one flat buffer so a step restarts with one copy
    Cflat = torch.empty_like(C0flat)
    views = list(torch.split(Cflat, sizes))
    for i, v in enumerate(views):
        st.C[i] = v.view(-1, 9)
        st.layers[i].C = st.C[i].data_ptr()
    bits = [kq.index_bits(L.k) for L in layers]
    cb_out = [(torch.empty(L.k * 9, dtype=torch.uint8, device=dev), torch.empty(64, device=dev),
               torch.empty(L.k, 9, device=dev)) for L in layers]
    p_idx = [torch.empty((L.n * b + 7) // 8 + 4, dtype=torch.uint8, device=dev) for L, b in zip(layers, bits)]
    p_codes = [torch.empty((L.k * 9 * 6 + 7) // 8 + 4, dtype=torch.uint8, device=dev) for L in layers]
    W_hat = [torch.empty(L.n, 9, device=dev) for L in layers]
    sq = torch.zeros(len(layers), dtype=torch.float64, device=dev)
    pack_jobs = [(st.idx[i], bits[i], p_idx[i]) for i in range(len(layers))] + \
                [(cb_out[i][0], 6, p_codes[i]) for i in range(len(layers))]
    recon = [{"packed": p_idx[i], "bits": bits[i], "n": L.n, "C": cb_out[i][2], "W_hat": W_hat[i], "W_ref": X[i],
              "sq_error": sq[i:i + 1]} for i, L in enumerate(layers)]
    recon_ws = torch.zeros(max(256, kq.recon_workspace_bytes(recon)), dtype=torch.uint8, device=dev)

    # the member sums come with the assignment when every codebook fits the fused variant
    fused = max(L.k for L in layers) <= 256 and not args.unfused
    stream = torch.cuda.current_stream(dev)
    ev = {"assign": [], "assign_final": [], "update": [], "cbq": [], "pack": [], "reconstruct": [], "fit": []}
    if args.yinyang:
        C0_views = [v.view(-1, 9) for v in torch.split(C0flat, sizes)]
        yy_ws = [torch.empty(kq.lib.kq_yinyang_workspace_bytes(L.n, L.k, 0), dtype=torch.uint8, device=dev)
                 for L in layers]
        yy_stats = [torch.zeros(max(T, 1), 3, dtype=torch.int64, device=dev) for L in layers]

    def timed(name, record, fn):
        if not record:
            fn()
            return
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        ev[name].append((e0, e1))

    def yinyang_rounds(record: bool):
        for i in range(len(layers)):
            timed("fit", record, lambda i=i: kq.kq_fit_layer_yinyang(
                X[i], C0_views[i], T, C=st.C[i], idx=st.idx[i], counts=st.counts[i],
                distortion=st.distortion[i], stats=yy_stats[i], workspace=yy_ws[i]))

    def step(record: bool):
        if args.yinyang:
            yinyang_rounds(record)
            timed("cbq", record, lambda: kq.kq_quantize_codebook_stack(st.C, st.counts, 6, kq.KQ_CBQ_WKMEANS, 30,
                                                                       out=cb_out))
            timed("pack", record, lambda: kq.kq_pack_bits_stack(pack_jobs))
            timed("reconstruct", record, lambda: kq.kq_reconstruct_stack(recon, workspace=recon_ws))
            return
        Cflat.copy_(C0flat)
        for t in range(T + 1):
            if record:
                a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a0.record(stream)
            kq.kq_assign_stack(st, dist_slot=t, distortion=False, fused_sums=fused and t < T)
            if record:
                a1.record(stream)
                # the rounds' launches (fused when the sums come with them) and the final one apart
                ev["assign" if t < T else "assign_final"].append((a0, a1))
            if t < T:
                if record:
                    u0, u1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    u0.record(stream)
                kq.kq_update_stack(st, dist_slot=t, distortion_from_assign=True, sums_from_assign=fused)
                if record:
                    u1.record(stream)
                    ev["update"].append((u0, u1))
        kq.kq_update_stack(st, dist_slot=T, counts_only=True, distortion_from_assign=True)
        timed("cbq", record, lambda: kq.kq_quantize_codebook_stack(st.C, st.counts, 6, kq.KQ_CBQ_WKMEANS, 30,
                                                                   out=cb_out))
        timed("pack", record, lambda: kq.kq_pack_bits_stack(pack_jobs))
        timed("reconstruct", record, lambda: kq.kq_reconstruct_stack(recon, workspace=recon_ws))

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(False)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = 1e3 * elapsed / args.steps
    # Per-launch durations: one more step with HIP events around every launch on the stream
    # the kernels run on.  It is kept out of the timed steps above because an event record
    # between two kernels adds a few microseconds of its own to the step.  Two untimed steps
    # are queued first: the host then enqueues the event step while the GPU still works
    # through them, so every event is stamped by the GPU's progress and not by a host that
    # is slower than the kernels it launches.
    for _ in range(2):
        step(False)
    step(True)
    torch.cuda.synchronize()

    # Eq. (2) codebook retraining step on the same stack (not part of the step): synthetic
    # gradients of the kernels' shape, the final assignment, one launch set per step
    gst = kq.Stack([x * 1e-3 for x in X], [c.view(-1, 9) for c in st.C])
    for i in range(len(layers)):
        gst.idx[i].copy_(st.idx[i])
    kq.kq_codebook_grad_step_stack(gst, 0.01)
    step(False)  # queued GPU work ahead of the events, as above
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g0.record(stream)
    for _ in range(5):
        kq.kq_codebook_grad_step_stack(gst, 0.01)
    g1.record(stream)
    torch.cuda.synchronize()
    grad_ms = g0.elapsed_time(g1) / 5

    # reconstruction alone (int32 indices, no error; not part of the step): 4 B read and
    # 36 B written per kernel, five launches between HIP events after a queued step
    recon_plain = [{"idx": st.idx[i], "n": L.n, "C": cb_out[i][2], "W_hat": W_hat[i]} for i, L in enumerate(layers)]
    step(False)
    r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    r0.record(stream)
    for _ in range(5):
        kq.kq_reconstruct_stack(recon_plain, workspace=recon_ws)
    r1.record(stream)
    torch.cuda.synchronize()
    recon_plain_ms = r0.elapsed_time(r1) / 5

    if args.copy_probe > 0:
        src = torch.ones(args.copy_probe << 18, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    mean_ms = {name: float(np.mean([a.elapsed_time(b) for a, b in pairs])) if pairs else 0.0
               for name, pairs in ev.items()}
    assign_ms, update_ms = mean_ms["assign"], mean_ms["update"]
    rec_bytes = sum(L.n * (b / 8 + 36 + 36) for L, b in zip(layers, bits))  # packed index + reference + output row
    flops = 18.0 * sum(L.k * L.n for L in layers)   # 9 multiply-adds per (kernel, entry) pair
    achieved = flops / (assign_ms * 1e-3) / 1e12 if assign_ms > 0 else 0.0
    # the separate update reads a 36-byte kernel and a 4-byte index per kernel; with fused
    # sums the round's update is only the finish over the assignment's partial sums, so no
    # kernel bytes are credited to it
    upd_bytes = 40.0 * n_total
    upd_gbs = upd_bytes / (update_ms * 1e-3) / 1e9 if update_ms > 0 and not fused else None

    yy_diag = None
    if args.yinyang:
        # the fits' own work: the round-0 assignment is a full one (n k distances), rounds
        # 1..T scan what the bounds leave (per-round counts from the library)
        stats = [s.cpu().numpy() for s in yy_stats]
        evals = sum(L.n * L.k + int(s[:T, 2].sum()) for L, s in zip(layers, stats))
        full = sum(L.n * L.k * (T + 1) for L in layers)
        fit_ms = sum(a.elapsed_time(b) for a, b in ev["fit"])
        yy_diag = {"fit_ms": fit_ms, "distance_evaluations": evals, "lloyd_equivalent": full,
                   "evaluated_fraction": evals / full,
                   "kernels_scanned_per_round": [int(x) for x in np.sum([s[:T, 0] for s in stats], axis=0)],
                   "pairs_scanned_per_round": [int(x) for x in np.sum([s[:T, 1] for s in stats], axis=0)]}
        achieved = 18.0 * evals / (fit_ms * 1e-3) / 1e12
    J = [float(d[T]) for d in st.distortion]
    mse_k = [j / (9 * L.n) for j, L in zip(J, layers)]
    mse_kc = [float(s) / (9 * L.n) for s, L in zip(sq.cpu(), layers)]
    print(json.dumps({"diag": {
        "assign_ms": assign_ms, "assign_TFLOPs": achieved, "update_ms": update_ms, "update_is_finish_only": fused,
        "update_GBps": upd_gbs,
        "lloyd_round_ms": assign_ms + update_ms, "final_assign_ms": mean_ms["assign_final"], "cbq_ms": mean_ms["cbq"], "pack_ms": mean_ms["pack"],
        "reconstruct_ms": mean_ms["reconstruct"],
        "reconstruct_GBps": rec_bytes / (mean_ms["reconstruct"] * 1e-3) / 1e9 if mean_ms["reconstruct"] else 0.0,
        "reconstruct_plain_ms": recon_plain_ms,
        "reconstruct_plain_GBps": 40.0 * n_total / (recon_plain_ms * 1e-3) / 1e9,
        "grad_step_ms": grad_ms, "grad_step_GBps": 40.0 * n_total / (grad_ms * 1e-3) / 1e9,
        "mse_K_first_last": [mse_k[0], mse_k[-1]], "mse_KC_first_last": [mse_kc[0], mse_kc[-1]],
        "beta_K": sum(L.k * 9 * 32 + L.n * b for L, b in zip(layers, bits)) / (9 * n_total),
        "beta_KC": sum(L.k * 9 * 6 + L.n * b for L, b in zip(layers, bits)) / (9 * n_total),
        "yinyang": yy_diag}}), file=sys.stderr)

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
                               "6-bit weighted codebook quantization, index/code packing, packed reconstruction",
                   "layers": len(layers), "kernels": n_total, "k": k, "lloyd_rounds": T, "codebook_bits": 6},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / FP32_PEAK_TFLOPS,
                     "traffic": assign_traffic() if (args.config, k) == ("resnet18", 256) and fused else None,
                     "kernel": ("assign_kernel<2, true> (member sums fused)" if fused else "assign_kernel<2, false>")
                               + " averaged over the Lloyd rounds' launches (one per round, whole stack)"},
    }
    if args.yinyang:
        # distances the Yinyang fits evaluated (matrix-core round 0 + exact fp32 scans), 18 flop
        # each, over the fits' whole time (updates included); the scans run unpacked fp32 VALU
        result["config"]["assignment"] = "yinyang"
        result["roofline"] = {"bound": "alu", "achieved": achieved, "peak": FP32_PEAK_TFLOPS / 2, "unit": "TFLOP/s",
                              "frac": achieved / (FP32_PEAK_TFLOPS / 2), "traffic": None,
                              "kernel": "kq_fit_layer_yinyang (all launches of the fits)"}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(layers, args.cpu_iters)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
