"""Throughput of Turbo-Muon orthogonalization (AOL + 4 quintic Newton-Schulz
iterations) on one MI355X, through the C ABI of libturbomuon.so.

One step = one tm_orthogonalize call over a batch of synthetic gradient-like
matrices already resident in HBM (default: 8 bf16 4096 x 14336 matrices,
power-law spectrum k^-0.5 plus 0.01 Gaussian noise).  The batch is updated in
place, so step i+1 orthogonalizes the output of step i; the kernels' work does
not depend on the values.  Prints one JSON line.
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

WORKLOADS = {
    # name: (count, m, n, alpha, dtype)
    "llm8b_4096x14336_b8": (8, 4096, 14336, 0.5, "bf16"),
    "llm8b_4096x4096_b8": (8, 4096, 4096, 0.5, "bf16"),
    "gpt2_mlp_768x3072": (1, 768, 3072, 0.8, "bf16"),
}


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
    ap.add_argument("--workload", default="llm8b_4096x14336_b8", choices=sorted(WORKLOADS))
    ap.add_argument("--iters", type=int, default=4)
    ap.add_argument("--precond", default="aol", choices=["aol", "frobenius", "none"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-check", action="store_true")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="after the timed region, run one plain device copy of this many MiB "
                         "(reference kernel for scaling the FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--inputs", default="powerlaw", choices=["powerlaw", "gaussian"],
                    help="powerlaw: the seeded power-law-plus-noise recipe (QR on the GPU); "
                         "gaussian: i.i.d. N(0,1) entries, the paper's own synthetic law "
                         "(for counter runs, where the QR library is not wanted)")
    args = ap.parse_args(argv)
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (asked for --gpus {args.gpus}); "
              "matrices are independent and would be sharded by count across GPUs, "
              "which is not built here.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2512_04632_amd import _lib as tm
    from paper_2512_04632_amd import synth

    count, m, n, alpha, dtype = WORKLOADS[args.workload]
    k, N = min(m, n), max(m, n)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    def progress(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    progress(f"generating {count} x {m}x{n} {dtype} alpha={alpha}")
    if args.inputs == "powerlaw":
        X = synth.power_law_batch_device(count, m, n, alpha, seed=0, device=dev)
    else:
        g = torch.Generator(device=dev)
        g.manual_seed(0)
        X = torch.randn((count, m, n), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    torch.cuda.synchronize()
    x0_host = X[0].float().cpu().numpy().astype(np.float64)   # oracle input (exact bf16 values)

    # One checked call from the pristine input: matrix 0 against the oracle.
    check = {}
    out0 = None
    if not args.no_check:
        Xc = X[:1].clone()
        tm.orthogonalize(Xc, args.iters, None, args.precond)
        torch.cuda.synchronize()
        out0 = Xc[0].float().cpu().numpy().astype(np.float64)
        del Xc

    progress(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        tm.orthogonalize(X, args.iters, None, args.precond)
    torch.cuda.synchronize()

    tm.timing_reset()
    tm.timing_enable(True)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for _ in range(args.steps):
        tm.orthogonalize(X, args.iters, None, args.precond)
    stop.record(stream)
    torch.cuda.synchronize()
    tm.timing_enable(False)
    elapsed_ms = start.elapsed_time(stop)
    phases = {p: tm.timing_read(p) for p in ("gram", "aol_vector", "poly", "update", "frob")}
    progress(f"timed {args.steps} steps: {elapsed_ms:.3f} ms")

    ms_per_step = elapsed_ms / args.steps
    fl = alg_flops(k, N, args.iters)
    step_flops = fl["total"] * count
    tflops = step_flops / (ms_per_step * 1e-3) / 1e12
    upd_ms, upd_n = phases["update"]
    upd_avg_ms = upd_ms / max(upd_n, 1)
    upd_flops_per_launch = fl["update_per_iter"] * count
    upd_tflops = upd_flops_per_launch / (upd_avg_ms * 1e-3) / 1e12

    result = {
        "metric": "orthogonalized matrices/s (AOL + 4 NS iterations)",
        "value": round(count * args.steps / (elapsed_ms * 1e-3), 3),
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
        "config": {"workload": args.workload, "matrices": count, "m": m, "n": n,
                   "alpha": alpha, "iters": args.iters, "precond": args.precond},
        "tflops_algorithmic": round(tflops, 2),
        "pct_bf16_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2),
        "phase_ms_per_step": {p: round(v[0] / args.steps, 4) for p, v in phases.items()},
        "roofline": {"bound": "mfma", "kernel": "k_update",
                     "achieved": round(upd_tflops, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(upd_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": None,
                     "launch_avg_ms": round(upd_avg_ms, 4),
                     "flops_per_launch": upd_flops_per_launch},
    }

    if out0 is not None or not args.no_cpu_baseline:
        from oracle import turbomuon as O
        t0 = time.perf_counter()
        ref0 = O.orthogonalize(x0_host, args.iters, None, args.precond)
        cpu_s = time.perf_counter() - t0
        if out0 is not None:
            check = {"rel_frobenius_vs_oracle": float(O.rel_frobenius(out0, ref0)),
                     "eps_ortho_gpu": float(O.eps_ortho(out0)),
                     "eps_ortho_oracle": float(O.eps_ortho(ref0)),
                     "matrix": 0}
            result["parity"] = check
        if not args.no_cpu_baseline:
            try:
                from threadpoolctl import threadpool_info
                cores = max(int(i.get("num_threads", 1)) for i in threadpool_info()) or 1
            except Exception:  # noqa: BLE001
                cores = os.cpu_count() or 1
            result["cpu_baseline"] = {"value": round(1.0 / cpu_s, 5), "unit": "matrices/s",
                                      "cores": cores, "kind": "oracle",
                                      "sample": f"1 of the {count} matrices ({m}x{n}), "
                                                f"fp64 NumPy, {cpu_s:.2f} s"}
    if args.copy_calibration_mb > 0:
        nbytes = args.copy_calibration_mb << 20
        src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = nbytes

    traffic = _recorded_traffic(upd_flops_per_launch)
    if traffic is not None:
        result["roofline"]["traffic"] = traffic
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
