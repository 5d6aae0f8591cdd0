"""Benchmark of the forward-only ZO step on one MI355X.

Workload (default, `single_linear_4096`): one adapted linear layer in bf16,
d_in = d_out = 4096, rank r = 32, 8192 tokens per perturbation half, activations
with a planted low-rank structure (64 directions carrying 90% of the variance),
W ~ N(0, 0.02^2).  One step is the whole hot path of a +/- ZO step:
    P = x U (both halves)  ->  fused +/- adapted GEMM (C +/- eps Z formed in-kernel)
    ->  MSE of both halves against a fixed in-subspace teacher  ->  ZO-Adam on C.
The activation basis U comes from the one-shot basis initialisation (timed
separately, outside the step).  Inputs are resident in HBM before timing starts.

Prints one JSON line: steps/s, ms/step, the roofline entry of the dominant kernel
(the fused GEMM: algorithmic FLOPs per launch / its mean duration measured with
HIP events on its stream, against the 2.5 PFLOP/s dense bf16 MFMA peak) and the
oracle's throughput on the host cores for the same workload.
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

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0


def gemm_source_hash() -> str:
    with open(os.path.join(ROOT, "paper_2607_01125_amd", "csrc", "k_gemm.hip"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_record(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None when
    the summary is missing or was taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get(f"{kernel}@{workload}")
    if not rec or rec.get("source_sha256_16") != gemm_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_baseline(T, K, N, r, steps=2):
    """The oracle (NumPy, float64 products, bf16 rounding emulated) on the same workload."""
    import numpy as np

    import synth
    from oracle import adam as oadam
    from oracle import linear as olin
    from oracle import loss as oloss
    from oracle import rng as orng

    x, q = synth.planted_lowrank(T, K, seed=0)
    x = synth.bf16_round(x)
    w = synth.bf16_round(synth.normal((N, K), 0.02, 0, 2))
    ut = synth.bf16_round(q[:, :r].T.copy())          # same shape as the initialised basis
    tgt = synth.bf16_round(synth.normal((T, N), 1.0, 0, 5))
    c = np.zeros(N * r, np.float32)
    m = np.zeros_like(c)
    v = np.zeros_like(c)
    xs = np.stack([x, x])
    t0 = time.perf_counter()
    for t in range(1, steps + 1):
        y = olin.adapted_linear_pm(xs, w, None, ut, c.reshape(N, r), 1e-3, 1, t, 0, 0, "bf16")
        g = oadam.projected_grad(oloss.mse(y[0], tgt), oloss.mse(y[1], tgt), 1e-3)
        c, m, v, _ = oadam.zo_adam(c, m, v, g, orng.gauss_range(1, t, 0, 0, N * r), oadam.adam_scalars(1e-4, t))
    dt = time.perf_counter() - t0
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count()
    return {"value": steps / dt, "unit": "ZO steps/s", "cores": cores, "kind": "oracle",
            "sample": f"{steps} full steps of the same workload ({T} tokens per half, d={K}, r={r}), "
                      f"NumPy float64 products with bf16 rounding emulated, {dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="single_linear_4096")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (the multi-GPU path is a "
              f"design, not a build)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2607_01125_amd import zoact as Z

    dev = torch.device("cuda:0")
    T, K, N, r = 8192, 4096, 4096, 32
    eps, lr, seed = 1e-3, 1e-4, 1

    # ---- synthetic inputs, resident in HBM
    x, q = synth.planted_lowrank(T, K, seed=0)
    xb = torch.from_numpy(synth.bf16_round(x)).to(dev).to(torch.bfloat16)
    x_pm = torch.cat([xb, xb], dim=0).contiguous()                 # [2][T][K], halves share x here
    w = torch.from_numpy(synth.bf16_round(synth.normal((N, K), 0.02, 0, 2))).to(dev).to(torch.bfloat16)
    # in-subspace teacher: Y = x (W + C* Q_r^T)^T, C* ~ N(0, 0.05^2), planted directions Q_r
    cstar = torch.from_numpy(synth.normal((N, r), 0.05, 0, 4)).to(dev)
    qr = torch.from_numpy(q[:, :r].copy()).to(dev)
    tgt = (xb.float() @ (w.float() + cstar @ qr.T).T).to(torch.bfloat16).contiguous()

    # ---- one-shot basis (Algorithm 1) on the calibration activations, timed separately
    ut = torch.empty(r, K, dtype=torch.bfloat16, device=dev)
    eigv = torch.empty(r, dtype=torch.float32, device=dev)
    ws_b = torch.empty(Z.basis_init_workspace_bytes(K, r), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    Z.basis_init(xb, r, ut, ws_b, eigvals=eigv)
    torch.cuda.synchronize()
    init_ms = (time.perf_counter() - t0) * 1e3
    del ws_b

    c = torch.zeros(N * r, dtype=torch.float32, device=dev)
    arena = Z.Arena(c, torch.zeros_like(c), torch.zeros_like(c))
    layer = Z.Linear(w, K, N, r, ut, 0)
    p = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev)
    y = torch.empty(2 * T, N, dtype=torch.bfloat16, device=dev)
    loss = torch.zeros(2, dtype=torch.float32, device=dev)
    ws_l = torch.empty(Z.loss_workspace_bytes(), dtype=torch.uint8, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()

    def zo_step(t, ev=None):
        pert = Z.Pert(seed, t, 0, eps)
        Z.project(x_pm, ut, p)
        if ev is not None:
            ev[0].record(stream)
        Z.linear_fwd_pm(layer, arena, x_pm, T, p, y, pert)
        if ev is not None:
            ev[1].record(stream)
        Z.mse_pm(y, tgt, loss, ws_l)
        Z.step(arena, loss, pert, Z.adam_desc(lr, t), status)

    for t in range(1, args.warmup + 1):
        zo_step(t)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for i in range(args.steps):
        zo_step(args.warmup + 1 + i, evs[i])
    stop.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    gemm_ms = sum(a.elapsed_time(b) for a, b in evs) / args.steps
    ms_per_step = total_ms / args.steps
    flops = 2 * (2 * T) * N * K + 2 * (2 * T) * K * r + 2 * (2 * T) * r * N   # base + projection + correction
    gemm_flops = 2 * (2 * T) * N * K + 2 * (2 * T) * r * N
    achieved = gemm_flops / (gemm_ms * 1e-3) / 1e12
    assert int(status.item()) == 0, "non-finite projected gradient"

    out = {
        "metric": "ZO steps/sec (±ε forwards + Adam) and adapted-linear TFLOP/s at 8B shapes",
        "value": round(1e3 / ms_per_step, 3),
        "unit": "ZO steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (planted low-rank activations, random-init W, seeded)",
        "config": {"workload": "single adapted linear, bf16, d_in=d_out=4096, r=32, 8192 tokens per ± half "
                               "(fused ± forward + projection + MSE + ZO-Adam)",
                   "tokens_per_half": T, "d_in": K, "d_out": N, "rank": r, "eps": eps,
                   "parallelism": "single GPU"},
        "adapted_linear_tflops": round(flops / (ms_per_step * 1e-3) / 1e12, 1),
        "basis_init_ms": round(init_ms, 1),
        "roofline": {"kernel": "gemm_pm_kernel (fused ± adapted GEMM)", "bound": "mfma",
                     "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": traffic_record("gemm_pm_kernel", args.workload),
                     "flops_per_launch": gemm_flops, "mean_launch_us": round(gemm_ms * 1e3, 1)},
        "losses": [float(v) for v in loss.cpu().numpy()],
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(T, K, N, r)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
