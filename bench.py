"""Throughput of Turbo-Muon orthogonalization (AOL + 4 quintic Newton-Schulz
iterations) on one MI355X, through the C ABI of libturbomuon.so.

One step = one library call over a workload of synthetic gradient-like
matrices already resident in HBM (default: one batched tm_orthogonalize call
on 8 bf16 4096 x 14336 matrices, power-law spectrum j^-0.5 plus 0.01 Gaussian
noise; workloads with several shapes use one tm_orthogonalize_grouped call).
The matrices are updated in place, so step i+1 orthogonalizes the output of
step i; the kernels' work does not depend on the values.  Prints one JSON line.
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

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix-core peak (published)
PEAK_F32_TFLOPS = 157.3
HBM_GBPS = 8000.0

# Workloads are the synthetic recipes of paper_2512_04632_amd.synth: a list of
# (count, m, n, alpha) entries in one storage dtype.  One-entry workloads run as
# one batched call, several entries as one grouped call.
DEFAULT_WORKLOAD = "llm8b_4096x14336_b8"
PRECOND_NAME = {"aol": "AOL", "frobenius": "Frobenius", "none": "no pre-conditioning"}


def alg_flops(k: int, N: int, iters: int) -> dict:
    """Algorithmic flops per matrix: symmetric products counted once per pair."""
    gram = k * (k + 1) * N            # upper triangle of Y Y^T
    poly = k * k * (k + 1) + 3 * k * k  # upper triangle of A A, plus the axpy
    update = 2 * k * k * N + 2 * k * N  # B Y plus a Y
    return {"gram": gram * iters, "poly": poly * iters, "update": update * iters,
            "total": (gram + poly + update) * iters, "update_per_iter": update}


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD,
                    help="one of paper_2512_04632_amd.synth.WORKLOADS")
    ap.add_argument("--iters", type=int, default=4)
    ap.add_argument("--precond", default="aol", choices=["aol", "frobenius", "none"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-check", action="store_true")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after the timed region, run one plain device copy of this many MiB "
                         "(reference kernel for scaling the FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--no-phase-timing", action="store_true",
                    help="leave the library's per-launch event hooks off in the timed region "
                         "(no phase split and no roofline figure; the step time then carries no "
                         "event-recording overhead, which matters for small workloads)")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step into a HIP graph (torch.cuda.graph, on a side "
                         "stream warmed up first) and time its replays; implies "
                         "--no-phase-timing")
    ap.add_argument("--optimizer", action="store_true",
                    help="time the optimizer step (tm_muon_step_grouped: momentum, bf16 "
                         "orthogonalization, fp32 parameter update) over the workload's matrices "
                         "instead of the orthogonalization alone")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-configuration sub-records that follow the default "
                         "workload's line (every other synthetic workload, timed the same way)")
    ap.add_argument("--inputs", default="powerlaw", choices=["powerlaw", "gaussian"],
                    help="powerlaw: the seeded power-law-plus-noise recipe (QR on the GPU); "
                         "gaussian: i.i.d. N(0,1) entries, the paper's own synthetic law "
                         "(for counter runs, where the QR library is not wanted)")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU only (asked for --gpus {args.gpus}); "
              "matrices are independent and would be sharded by count across GPUs, "
              "which is not built here.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2512_04632_amd import _lib as tm
    from paper_2512_04632_amd import synth

    if args.workload not in synth.WORKLOADS:
        print(f"bench.py: unknown workload {args.workload!r}; choose from "
              f"{sorted(synth.WORKLOADS)}", file=sys.stderr)
        return 2
    spec = synth.WORKLOADS[args.workload]
    dtype = spec["dtype"]
    entries = spec["entries"]
    tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
    grouped = len(entries) > 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    def progress(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    progress(f"generating {args.workload}: {entries} {dtype}")
    batches = []
    for e, (count, m, n, alpha) in enumerate(entries):
        if args.inputs == "powerlaw":
            X = synth.power_law_batch_device(count, m, n, alpha, seed=e, device=dev, dtype=tdtype)
        else:
            g = torch.Generator(device=dev)
            g.manual_seed(e)
            X = torch.randn((count, m, n), generator=g, device=dev, dtype=torch.float32).to(tdtype)
        batches.append(X)
    torch.cuda.synchronize()
    n_mat = sum(c for c, _, _, _ in entries)

    if args.optimizer:
        return _bench_optimizer(args, batches, entries, dev, stream, progress)

    def run(bs):
        if grouped:
            tm.orthogonalize_grouped([X[i] for X in bs for i in range(X.shape[0])], args.iters,
                                     None, args.precond)
        else:
            tm.orthogonalize(bs[0], args.iters, None, args.precond)

    # One checked call from the pristine inputs: matrix 0 of every entry
    # against the oracle, on the exact stored values.
    hosts = [X[0].float().cpu().numpy().astype(np.float64) for X in batches]
    outs = None
    if not args.no_check and not args.no_cpu_baseline:
        clones = [X.clone() for X in batches]
        run(clones)
        torch.cuda.synchronize()
        outs = [X[0].float().cpu().numpy().astype(np.float64) for X in clones]
        del clones

    progress(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        run(batches)
    torch.cuda.synchronize()

    step = lambda: run(batches)  # noqa: E731
    if args.graph:
        # The library keeps its workspace per (device, stream): one call on the
        # capture stream sizes it, so the captured call allocates nothing.
        args.no_phase_timing = True
        side = torch.cuda.Stream(dev)
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            run(batches)
        side.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            run(batches)
        torch.cuda.synchronize()
        for _ in range(max(1, args.warmup)):
            graph.replay()
        torch.cuda.synchronize()
        step = graph.replay
        progress("captured one step into a graph")

    tm.timing_reset()
    tm.timing_enable(not args.no_phase_timing)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    tm.timing_enable(False)
    elapsed_ms = start.elapsed_time(stop)
    phase_names = ("load_in", "frob", "gram", "aol_vector", "scale_a", "poly", "update", "fused")
    phases = {p: tm.timing_read(p) for p in phase_names}
    progress(f"timed {args.steps} steps: {elapsed_ms:.3f} ms")

    ms_per_step = elapsed_ms / args.steps
    step_flops = 0
    upd_flops_per_iter = 0
    for count, m, n, _ in entries:
        fl = alg_flops(min(m, n), max(m, n), args.iters)
        step_flops += fl["total"] * count
        upd_flops_per_iter += fl["update_per_iter"] * count
    tflops = step_flops / (ms_per_step * 1e-3) / 1e12
    upd_ms, upd_n = phases["update"]
    upd_avg_ms = upd_ms / upd_n if upd_n else None
    # a call with more than 64 matrices (or a split last wave) runs an
    # iteration's update as several launches: average over all of them
    upd_flops_total = upd_flops_per_iter * args.iters * args.steps
    upd_flops_per_launch = (upd_flops_total // upd_n if upd_n and upd_flops_total % upd_n == 0
                            else (upd_flops_total / upd_n if upd_n else 0))
    upd_tflops = upd_flops_total / (upd_ms * 1e-3) / 1e12 if upd_n else None
    peak = PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_F32_TFLOPS

    config = {"workload": args.workload, "matrices": n_mat,
              "shapes": [[c, m, n] for c, m, n, _ in entries],
              "alpha": [a for _, _, _, a in entries], "iters": args.iters,
              "precond": args.precond, "call": "grouped" if grouped else "batched"}
    if args.graph:
        config["launch"] = "hip graph replay"
    result = {
        "metric": f"orthogonalized matrices/s ({PRECOND_NAME[args.precond]} + {args.iters} NS iterations)",
        "value": round(n_mat * args.steps / (elapsed_ms * 1e-3), 3),
        "unit": "matrices/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": ("synthetic (seeded power-law spectrum + 0.01 Gaussian noise)"
                 if args.inputs == "powerlaw" else "synthetic (seeded i.i.d. N(0,1))"),
        "config": config,
        "tflops_algorithmic": round(tflops, 2),
        "pct_peak": round(100 * tflops / peak, 2),
        "phase_ms_per_step": {p: round(v[0] / args.steps, 4) for p, v in phases.items()},
        "roofline": {"bound": "mfma", "kernel": "k_update_fast",
                     "achieved": round(upd_tflops, 2) if upd_n else None, "peak": peak,
                     "unit": "TFLOP/s", "frac": round(upd_tflops / peak, 4) if upd_n else None,
                     "traffic": None,
                     "launch_avg_ms": round(upd_avg_ms, 4) if upd_n else None,
                     "launches": upd_n,
                     "flops_per_launch": upd_flops_per_launch,
                     "source": "HIP events recorded on the call's stream around every "
                               "k_update_fast launch of the timed steps (library timing hooks); "
                               "achieved = update flops of those launches / their summed time"},
    }
    fused_ms, fused_n = phases["fused"]
    if not upd_n and fused_n:
        # every phase and iteration of a call in one k_small_ns launch per call
        fl_fused = step_flops * args.steps / (fused_ms * 1e-3) / 1e12
        result["roofline"] = {
            "bound": "mfma", "kernel": "k_small_ns", "achieved": round(fl_fused, 2), "peak": peak,
            "unit": "TFLOP/s", "frac": round(fl_fused / peak, 4), "traffic": None,
            "launch_avg_ms": round(fused_ms / fused_n, 4), "launches": fused_n,
            "flops_per_launch": step_flops * args.steps // fused_n,
            "source": "HIP events recorded on the call's stream around every k_small_ns launch "
                      "of the timed steps (library timing hooks; one launch runs a whole call); "
                      "achieved = the calls' algorithmic flops / the launches' summed time"}

    if not args.no_cpu_baseline:
        # The cpu_baseline leg: the oracle timed on the host cores; its results
        # for matrix 0 of every entry also give the run's parity figures.
        from oracle import turbomuon as O
        refs, cpu_s = [], []
        for Xh in hosts:
            t0 = time.perf_counter()
            refs.append(O.orthogonalize(Xh, args.iters, None, args.precond))
            cpu_s.append(time.perf_counter() - t0)
        if outs is not None:
            result["parity"] = [{"entry": e, "matrix": 0,
                                 "rel_frobenius_vs_oracle": float(O.rel_frobenius(o, r)),
                                 "eps_ortho_gpu": float(O.eps_ortho(o)),
                                 "eps_ortho_oracle": float(O.eps_ortho(r))}
                                for e, (o, r) in enumerate(zip(outs, refs))]
        # Bounded sample: the oracle on the workload's matrices in order
        # (the first matrix of each entry already timed above, then more of
        # the first entry) until about 10 s of CPU time have been spent.
        done, spent = len(hosts), sum(cpu_s)
        X0 = batches[0]
        i = 1
        while spent < 10.0 and i < X0.shape[0]:
            Xh = X0[i].float().cpu().numpy().astype(np.float64)
            t0 = time.perf_counter()
            O.orthogonalize(Xh, args.iters, None, args.precond)
            spent += time.perf_counter() - t0
            done += 1
            i += 1
        try:
            from threadpoolctl import threadpool_info
            cores = max(int(i.get("num_threads", 1)) for i in threadpool_info()) or 1
        except Exception:  # noqa: BLE001
            cores = os.cpu_count() or 1
        result["cpu_baseline"] = {
            "value": round(done / spent, 5), "unit": "matrices/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{done} of the {n_mat} matrices, fp64 NumPy, {spent:.2f} s"}
    if args.copy_calibration_mb > 0:
        nbytes = args.copy_calibration_mb << 20
        src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = nbytes

    if not args.no_configs and args.workload == DEFAULT_WORKLOAD and not args.graph:
        result["configs"] = _config_records(args, dev, progress)

    traffic = _recorded_traffic(upd_flops_per_launch) if args.workload == DEFAULT_WORKLOAD else None
    if traffic is not None:
        result["roofline"]["traffic"] = traffic
    print(json.dumps(result), flush=True)
    return 0


# The other configurations of the benchmark's workload list, reported as
# sub-records of the default line: (label, workload, iters, precond).  The
# 4096 x 14336 half of the 8B-class configuration is the line itself.
CONFIGS = [
    ("single_256_f32", "single_256_f32", 4, "aol"),
    ("gpt2_mlp_768x3072", "gpt2_mlp_768x3072", 4, "aol"),
    ("gpt2_mlp_768x3072_muon", "gpt2_mlp_768x3072", 5, "frobenius"),
    ("gpt2_small_12layer", "gpt2_small_12layer", 4, "aol"),
    ("llm8b_4096x4096_b8", "llm8b_4096x4096_b8", 4, "aol"),
    ("resnet_conv_64", "resnet_conv_64", 4, "aol"),
    ("resnet_conv_64x576_b16", "resnet_conv_64x576_b16", 4, "aol"),
]


def _config_records(args, dev, progress):
    """Each configuration timed like the line (inputs resident in HBM, warm-up,
    then 20 timed calls on the current stream) but without the per-launch
    timing hooks, whose two event records per launch matter for the small
    workloads.  The oracle on matrix 0 of every shape of a configuration, on
    the host cores, is that configuration's CPU baseline and its parity
    figure (skipped with --no-cpu-baseline)."""
    import numpy as np
    import torch

    from paper_2512_04632_amd import _lib as tm
    from paper_2512_04632_amd import synth

    out = []
    steps, warmup = 20, 5
    stream = torch.cuda.current_stream(dev)
    for label, wl, iters, precond in CONFIGS:
        spec = synth.WORKLOADS[wl]
        dtype = spec["dtype"]
        tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        entries = spec["entries"]
        progress(f"config {label}: {wl} {precond} t={iters}")
        batches = [synth.power_law_batch_device(c, m, n, a, seed=e, device=dev, dtype=tdtype)
                   for e, (c, m, n, a) in enumerate(entries)]
        grouped = len(entries) > 1

        def run(bs):
            if grouped:
                tm.orthogonalize_grouped([X[i] for X in bs for i in range(X.shape[0])], iters,
                                         None, precond)
            else:
                tm.orthogonalize(bs[0], iters, None, precond)

        hosts = [X[0].float().cpu().numpy().astype(np.float64) for X in batches]
        clones = [X.clone() for X in batches]
        run(clones)
        torch.cuda.synchronize()
        outs = [X[0].float().cpu().numpy().astype(np.float64) for X in clones]
        del clones
        for _ in range(warmup):
            run(batches)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(steps):
            run(batches)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        # calls that the fused small-matrix kernel serves: the same calls on the
        # tiled kernels, for comparison
        tm.timing_reset()
        tm.timing_enable(True)
        run(batches)
        torch.cuda.synchronize()
        tm.timing_enable(False)
        fused = tm.timing_read("fused")[1] > 0
        tm.timing_reset()
        tiled_ms = None
        if fused:
            os.environ["TM_DISABLE_FUSED"] = "1"
            try:
                for _ in range(warmup):
                    run(batches)
                e0.record(stream)
                for _ in range(steps):
                    run(batches)
                e1.record(stream)
                torch.cuda.synchronize()
                tiled_ms = e0.elapsed_time(e1) / steps
            finally:
                del os.environ["TM_DISABLE_FUSED"]
        n_mat = sum(c for c, _, _, _ in entries)
        flops = sum(alg_flops(min(m, n), max(m, n), iters)["total"] * c for c, m, n, _ in entries)
        peak = PEAK_BF16_TFLOPS if dtype == "bf16" else PEAK_F32_TFLOPS
        rec = {"config": label, "workload": wl, "call": "grouped" if grouped else "batched",
               "shapes": [[c, m, n] for c, m, n, _ in entries], "dtype": dtype, "iters": iters,
               "precond": precond, "steps": steps, "ms_per_step": round(ms, 4),
               "matrices_per_s": round(n_mat / (ms * 1e-3), 2),
               "tflops_algorithmic": round(flops / (ms * 1e-3) / 1e12, 2),
               "pct_peak": round(100 * flops / (ms * 1e-3) / 1e12 / peak, 2),
               "kernels": "fused" if fused else "tiled"}
        if tiled_ms is not None:
            rec["tiled_ms_per_step"] = round(tiled_ms, 4)
        if not args.no_cpu_baseline:
            # cpu_baseline leg of this configuration: the oracle on matrix 0 of
            # every shape, timed on the host cores; its results give the parity
            from oracle import turbomuon as O
            par, spent = [], 0.0
            for e, (Xh, G) in enumerate(zip(hosts, outs)):
                t0 = time.perf_counter()
                R = O.orthogonalize(Xh, iters, None, precond)
                spent += time.perf_counter() - t0
                item = {"entry": e, "matrix": 0,
                        "rel_frobenius_vs_oracle": float(O.rel_frobenius(G, R)),
                        "eps_ortho_gpu": float(O.eps_ortho(G)),
                        "eps_ortho_oracle": float(O.eps_ortho(R))}
                if label == "single_256_f32":   # the accuracy configuration: distance to the SVD polar factor
                    Q = O.polar_factor(Xh)
                    item["eps_polar_gpu"] = float(O.eps_polar(G, Xh, Q))
                    item["eps_polar_oracle"] = float(O.eps_polar(R, Xh, Q))
                par.append(item)
            rec["parity"] = par
            rec["cpu_baseline"] = {"value": round(len(hosts) / spent, 4), "unit": "matrices/s",
                                   "kind": "oracle",
                                   "sample": f"matrix 0 of each of the {len(hosts)} shapes, "
                                             f"fp64 NumPy, {spent:.2f} s"}
        out.append(rec)
        del batches
        torch.cuda.empty_cache()
    tm.release_workspaces()
    return out


def _bench_optimizer(args, batches, entries, dev, stream, progress):
    """Optimizer steps/s over fp32 parameters shaped like the workload's matrices."""
    import torch

    from paper_2512_04632_amd import _lib as tm
    g = torch.Generator(device=dev)
    g.manual_seed(1)
    grads = [X[i].float().contiguous() for X in batches for i in range(X.shape[0])]
    params = [0.02 * torch.randn(t.shape, generator=g, device=dev) for t in grads]
    bufs = [torch.zeros_like(t) for t in grads]
    lr, mu = 0.02, 0.95

    def step():
        tm.muon_step_grouped(params, grads, bufs, lr, mu, True, 0.0, True, args.iters, None,
                             args.precond)

    progress(f"optimizer warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    tm.timing_reset()
    tm.timing_enable(True)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    tm.timing_enable(False)
    ms = start.elapsed_time(stop) / args.steps
    names = ("opt_momentum", "load_in", "gram", "aol_vector", "scale_a", "poly", "update",
             "opt_apply")
    phases = {p: round(tm.timing_read(p)[0] / args.steps, 4) for p in names}
    n_el = sum(t.numel() for t in grads)
    result = {
        "metric": f"optimizer steps/s ({PRECOND_NAME[args.precond]} + {args.iters} NS iterations)",
        "value": round(1e3 / ms, 3), "unit": "steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32 parameters, bf16 orthogonalization",
        "data": "synthetic (seeded power-law gradients, N(0, 0.02^2) parameters)",
        "config": {"workload": args.workload, "matrices": len(grads), "parameters": n_el,
                   "shapes": [[c, m, n] for c, m, n, _ in entries], "lr": lr, "momentum": mu,
                   "nesterov": True},
        "phase_ms_per_step": phases,
        "elementwise_gbps": round((14 + 10) * n_el / ((phases["opt_momentum"] + phases["opt_apply"])
                                                      * 1e-3) / 1e9, 1)
        if phases["opt_momentum"] + phases["opt_apply"] > 0 else None,
    }
    print(json.dumps(result), flush=True)
    return 0


def _recorded_traffic(flops_per_launch):
    """HBM bytes per k_update_fast launch from the committed counter summary.

    The summary records the hash of the kernel source it was taken with; a
    changed kernel reports null.
    """
    import hashlib
    path = os.path.join(ROOT, "profiles", "k_update_fast_traffic.json")
    src = os.path.join(ROOT, "paper_2512_04632_amd", "csrc", "tm_fast.hip")
    try:
        with open(path) as f:
            rec = json.load(f)
        with open(src, "rb") as f:
            h = hashlib.sha256(f.read()).hexdigest()
    except OSError:
        return None
    if rec.get("kernel_source_sha256") != h or rec.get("flops_per_launch") != flops_per_launch:
        return None
    return rec.get("hbm_bytes_per_launch")


if __name__ == "__main__":
    sys.exit(main())
