"""Benchmark of the forward-only ZO step on one MI355X.

Headline workload (`llama3_8b_bf16_step`): one two-sided ZO step of a random-initialised
Llama-3-8B-shaped decoder in bf16 -- 32 layers, d = 4096, 32 query / 8 key-value heads of
128, SwiGLU FFN 14336, vocabulary 128256, rank r = 32 on all seven projections, 16 x 256
uniform random tokens per perturbation half, eps = 1e-3, Adam lr = 5e-5.  One step is the
whole hot path: both halves' forward with every adapted linear as one fused +/- GEMM (the
perturbed coefficients C +/- eps Z read from the previous update pass), the LM head with
the next-token cross entropy in its epilogue, then ZO-Adam on the 44,040,192 coefficients
(whose pass also forms the next step's C +/- eps Z).  The basis (Algorithm 1 on 16 x 256
calibration tokens) is computed before timing and reported separately.  Inputs and
weights are resident in HBM before the timed region starts.

`roofline` is the fused +/- adapted GEMM (`gemm_4w64_kernel`) over every adapted-linear
launch of the timed steps: algorithmic FLOPs per launch (2 M N K + 2 M r N, M = 2 x 4096
stacked rows; the shared first projection 2 T N K + 2 M r N) over the mean launch duration,
both from HIP events recorded around each launch on its stream, against the 2.5 PFLOP/s
dense bf16 MFMA peak.

Besides the headline the run measures (unless --quick): the single adapted linear
(4096 x 4096, r = 32, 8192 tokens per half) in its stacked and shared-input forms; the
fused +/- adapted linear at the Llama-3-8B layer shapes (bf16, INT4 in-register, INT4 via
the dequantisation pass) and across ranks; the INT4 Llama step; the OPT-13B-shape step with
its basis initialisation; ZO-Adam's HBM rate over the Llama arena; the one-sided q = 8 form;
the tiny fp32 model's 20 steps.  `cpu_baseline` is the oracle timed on the host cores on a
bounded sample of the headline step, extrapolated to a whole step; without --quick the same
kind of sample is taken for the INT4 and OPT-13B-shape steps (`models[...].cpu_baseline`) and
for Algorithm 1 over the Llama and OPT sites (`cpu_baseline_basis_init`).

Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
METRIC = "ZO steps/sec (±ε forwards + Adam) and adapted-linear TFLOP/s at 8B shapes"
DOMINANT_KERNEL = "gemm_4w64_kernel"
DOMINANT_SOURCES = [os.path.join("paper_2607_01125_amd", "csrc", f)
                    for f in ("k_gemm_4w64.hip", "gemm_4w_epi.hpp", "gemm_common.hpp")]
HEADLINE = "llama3_8b_bf16_step"
_LLAMA_TXT = ("32 layers, d=4096, GQA 32q/8kv x 128, SwiGLU FFN 14336, vocab 128256; r=32 on q,k,v,o,gate,up,down; "
              "16x256 tokens per ± half")
# workloads bench.py can time as its line (the headline by default; the others for profiling)
WORKLOADS = {
    HEADLINE: ("llama_bf16", "Llama-3-8B-shape decoder, bf16, random init: " + _LLAMA_TXT + "; one two-sided ZO step "
               "(± forward with the fused LM head + cross entropy, ZO-Adam over 44,040,192 coefficients)",
               {"tokens_per_half": 4096, "rank": 32, "eps": 1e-3, "lr": 5e-5}),
    "llama3_8b_int4_step": ("llama_int4", "Llama-3-8B-shape decoder, INT4 weights (groups of 128 along the input, "
                            "bf16 scales), bf16 activations, random init: " + _LLAMA_TXT + "; one two-sided ZO step",
                            {"tokens_per_half": 4096, "rank": 32, "eps": 1e-3, "lr": 5e-5}),
    "opt13b_bf16_step": ("opt_bf16", "OPT-13B-shape decoder, bf16, random init: 40 layers, d=5120, 40 heads x 128, "
                         "ReLU FFN 20480, vocab 50272, learned positions; r=64 on q,v,o,fc1,fc2; 8x512 tokens per ± "
                         "half; one two-sided ZO step", {"tokens_per_half": 4096, "rank": 64, "eps": 1e-3,
                                                         "lr": 2.5e-5}),
}


class TimingEvent:
    """A HIP timing event created with hipEventDisableSystemFence, recorded on a torch stream.

    Recording torch's events applies a system-scope release (cache writeback and
    invalidation), which put about 6 µs of idle time before the next kernel of a step;
    without the fence the events that bracket one launch add no gap to the step.  The
    HIP runtime is the one torch has loaded (this library resolves to the same one)."""

    _hip = None
    DISABLE_SYSTEM_FENCE = 0x20000000

    @classmethod
    def _rt(cls):
        if cls._hip is None:
            import ctypes

            path = None
            with open("/proc/self/maps") as f:
                for line in f:
                    if "libamdhip64.so" in line:
                        path = line.split()[-1]
                        break
            if path is None:
                raise RuntimeError("HIP runtime not loaded")
            h = ctypes.CDLL(path)
            h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._hip = h
        return cls._hip

    def __init__(self):
        import ctypes

        self._ev = ctypes.c_void_p()
        if self._rt().hipEventCreateWithFlags(ctypes.byref(self._ev), self.DISABLE_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream):
        if self._rt().hipEventRecord(self._ev, ctypes_stream(stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, end) -> float:
        import ctypes

        ms = ctypes.c_float()
        if self._rt().hipEventElapsedTime(ctypes.byref(ms), self._ev, end._ev) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        if self._hip is not None and self._ev:
            self._hip.hipEventDestroy(self._ev)


def ctypes_stream(stream):
    import ctypes

    return ctypes.c_void_p(stream.cuda_stream)


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def source_hash(rels) -> str:
    """Hash of the code in the given sources: comments, trailing blanks and empty lines are
    dropped, so a record taken on a kernel stays valid through comment edits."""
    h = hashlib.sha256()
    for rel in rels:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
        for line in text.splitlines():
            code = line.split("//", 1)[0].rstrip()
            if code:
                h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def traffic_record(kernel: str, workload: str, sources):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or None when
    the summary is missing or was taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get(f"{kernel}@{workload}")
    if not rec or rec.get("source_sha256_16") != source_hash(sources):
        return None
    return rec.get("hbm_bytes_per_launch")


# ------------------------------------------------------------------ CPU baseline (the oracle)
def _host_cores():
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count()
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    threads = cores
    try:
        from threadpoolctl import threadpool_info
        blas = [i["num_threads"] for i in threadpool_info() if i.get("user_api") == "blas"]
        if blas:
            threads = max(blas)
    except Exception:
        pass
    return cores, threads, model


_ORACLE_WEIGHTS = {}


def _oracle_forward_sample(full, B, S, n_seq, int4=False):
    """Times the oracle on one half's loss of a one-layer full-width model of `full` over
    n_seq of B sequences of S tokens, once with the full vocabulary and once with an 8-token
    head.  Returns (t_layer, t_full, gen_s, dq_s): t_layer (the 8-token-head run) holds the
    layer plus the embedding and the final norm, t_full - t_layer the LM head; gen_s is the
    untimed weight generation, dq_s the oracle's INT4 dequantisation of the layer's weights
    (done once, when the model is built, so not part of a step)."""
    import dataclasses as dc

    import numpy as np

    import synth
    from oracle import linear as olin
    from oracle import model as om

    shape = synth.shrink(full, n_layers=1)
    t_gen = time.perf_counter()
    if full.name not in _ORACLE_WEIGHTS:   # the headline and INT4 samples share one draw
        _ORACLE_WEIGHTS[full.name] = synth.model_weights(shape, 0, "bf16")
    W = dict(_ORACLE_WEIGHTS[full.name])
    gen_s = time.perf_counter() - t_gen
    dq_s = 0.0
    if int4:
        L = dict(W[0])
        for name in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "w1", "w2"):
            if name in L:
                packed, scales = synth.quantize_int4_g128(L[name])
                t0 = time.perf_counter()
                L[name] = olin.dequant_int4(packed, scales).astype(np.float32)
                dq_s += time.perf_counter() - t0
        W[0] = L
    small = dc.replace(shape, vocab=8)
    Ws = dict(W)
    for key in ("emb", "head"):
        if key in W:
            Ws[key] = W[key][:8].copy()
    tok = synth.uniform_tokens(B, S, full.vocab, 0, 2)[:n_seq]
    m_full = om.Model(shape, 0, "bf16", weights=W)
    m_small = om.Model(small, 0, "bf16", weights=Ws)
    d = full.d_model
    for m in (m_full, m_small):
        for key, d_in in {(0, "attn"): d, (0, "o"): d, (0, "mlp"): d, (0, "down"): full.d_ff}.items():
            q, _ = np.linalg.qr(synth.gen(0, 881, d_in).standard_normal((d_in, full.rank)))
            m.U[key] = q.astype(np.float32).astype(np.float64)
    c = np.zeros(m_full.k, np.float32)
    t0 = time.perf_counter()
    m_small.loss(tok % 8, c, +1, 1e-3, (1, 1, 0))
    t_layer = time.perf_counter() - t0
    t0 = time.perf_counter()
    m_full.loss(tok, c, +1, 1e-3, (1, 1, 0))
    t_full = time.perf_counter() - t0
    return t_layer, t_full, gen_s, dq_s


def _oracle_adam_sample(n_adam=4_194_304):
    """Seconds of the oracle's ZO-Adam (Gaussians regenerated) over n_adam coefficients."""
    import numpy as np

    from oracle import adam as oadam
    from oracle import rng as orng

    ca = np.zeros(n_adam, np.float32)
    t0 = time.perf_counter()
    z = orng.gauss_range(1, 1, 0, 0, n_adam)
    oadam.zo_adam(ca, ca, ca, 0.25, z, oadam.adam_scalars(5e-5, 1))
    return time.perf_counter() - t0


def _oracle_step_record(full, B, S, n_seq, what, int4=False):
    """The oracle's two-sided ZO step on `full`, sampled and extrapolated (see
    cpu_baseline_llama for the model of the step time)."""
    from oracle import model as om

    t_layer, t_full, gen_s, dq_s = _oracle_forward_sample(full, B, S, n_seq, int4)
    t_head = max(t_full - t_layer, 0.0)
    n_adam = 4_194_304
    t_adam = _oracle_adam_sample(n_adam)
    k = om.arena_size(full)
    scale = B // n_seq
    L = full.n_layers
    step_s = 2 * scale * (L * t_layer + t_head) + (k / n_adam) * t_adam
    cores, threads, model = _host_cores()
    rec = {"value": round(1.0 / step_s, 7), "unit": "ZO steps/s", "cores": threads, "kind": "oracle",
           "extrapolated": True, "cpu_model": model, "cores_available": cores,
           "seconds_per_step": round(step_s, 1),
           "sample": (f"one half's loss of a one-layer full-width {what} on {n_seq} of {B} "
                      f"sequences of {S} tokens, with the {full.vocab}-token head ({t_full:.2f} s) and with an "
                      f"8-token head ({t_layer:.2f} s), plus ZO-Adam with regenerated Gaussians over {n_adam} "
                      f"coefficients ({t_adam:.2f} s); extrapolated as 2 halves x {scale} x ({L} layers x "
                      f"{t_layer:.2f} s + head {t_head:.2f} s) + {k / n_adam:.1f} x {t_adam:.2f} s = "
                      f"{step_s:.0f} s per step; NumPy float64 products with the bf16 rounding points "
                      f"emulated (weights generated untimed in {gen_s:.0f} s)")}
    if int4:
        rec["int4_dequant_s"] = round(L * dq_s, 1)
        rec["sample"] += (f"; the oracle dequantises the INT4 weights once when the model is built "
                          f"({dq_s:.2f} s for the layer, {L * dq_s:.0f} s for {L} layers; not in the step)")
    return rec


def cpu_baseline_llama():
    """The oracle (NumPy, float64 products, bf16 rounding points emulated) on a bounded
    sample of the headline step, extrapolated to one whole step.

    A step is L+ and L- (each: embedding, 32 layers, final norm, LM head, cross entropy over
    16 x 256 tokens) and ZO-Adam over k = 44,040,192 coefficients.  Timed: one half's loss of
    a one-layer model at full width on 4 of the 16 sequences, once with the full vocabulary
    and once with an 8-token head; and the Adam update (Gaussians regenerated) over 4,194,304
    coefficients.  Every step of the oracle is per sequence, per layer or per coefficient, so
    the step time is  2 halves x 4 x (32 x t_layer + t_head) + (k / 4,194,304) x t_adam  with
    t_layer the 8-token-head time (it also holds the embedding and the final norm) and t_head
    the difference of the two."""
    import synth

    return _oracle_step_record(synth.LLAMA3_8B, 16, 256, 4, "Llama-3-8B-shape model")


def cpu_baseline_model(w):
    """The oracle's step for the side workloads, sampled as for the headline: the INT4
    Llama-3-8B shape (weights dequantised by the oracle) on 4 of 16 sequences of 256 tokens,
    the OPT-13B shape on 1 of 8 sequences of 512 tokens."""
    import synth

    if w == "llama_int4":
        return _oracle_step_record(synth.LLAMA3_8B, 16, 256, 4, "INT4 Llama-3-8B-shape model", int4=True)
    return _oracle_step_record(synth.OPT_13B, 8, 512, 1, "OPT-13B-shape model")


def cpu_baseline_basis(full, calib_tokens, t_sample=2048):
    """The oracle's Algorithm 1 (float64 Gram X^T X, then the top-r eigenvectors) over every
    adapted site of `full`, sampled on one site of width d_model: the Gram of t_sample
    calibration rows, and the eigensolve of a d_model x d_model Gram.  Extrapolated per site
    as  t_gram x (calib_tokens / t_sample) x (d / d_model)^2 + t_eig x (d / d_model)^3  (the
    Gram's cost is linear in the rows and quadratic in the width; the dense symmetric
    eigensolver's reduction is cubic in the width)."""
    import numpy as np

    import synth
    from oracle import basis as obasis

    d = full.d_model
    x = synth.bf16_round(synth.gen(0, 882, d).standard_normal((t_sample, d)).astype(np.float32))
    t0 = time.perf_counter()
    g = obasis.gram(x)
    t_gram = time.perf_counter() - t0
    t0 = time.perf_counter()
    obasis.top_eigvecs(g, full.rank)
    t_eig = time.perf_counter() - t0
    widths = [d, d, d, full.d_ff] * full.n_layers
    total = sum(t_gram * (calib_tokens / t_sample) * (w / d) ** 2 + t_eig * (w / d) ** 3 for w in widths)
    cores, threads, model = _host_cores()
    return {"value": round(total, 1), "unit": "s", "cores": threads, "kind": "oracle", "extrapolated": True,
            "cpu_model": model,
            "sample": (f"Algorithm 1 on one width-{d} site: the float64 Gram of {t_sample} rows "
                       f"({t_gram:.2f} s) and the top-{full.rank} eigenvectors of the {d} x {d} Gram "
                       f"({t_eig:.2f} s); extrapolated to the {len(widths)} sites (widths {d} and {full.d_ff}) "
                       f"and {calib_tokens} calibration tokens as t_gram x (tokens / {t_sample}) x (width / {d})^2 "
                       f"+ t_eig x (width / {d})^3 per site = {total:.0f} s")}


def cpu_baseline_single(T, K, N, r, budget_s=8.0):
    """The oracle on the single-layer workload (stacked form): whole steps until about
    `budget_s` seconds of host time have been spent."""
    import numpy as np

    import synth
    from oracle import adam as oadam
    from oracle import linear as olin
    from oracle import loss as oloss
    from oracle import rng as orng

    x, q = synth.planted_lowrank(T, K, seed=0)
    x = synth.bf16_round(x)
    w = synth.bf16_round(synth.normal((N, K), 0.02, 0, 2))
    ut = synth.bf16_round(q[:, :r].T.copy())
    tgt = synth.bf16_round(synth.normal((T, N), 1.0, 0, 5))
    c = np.zeros(N * r, np.float32)
    m = np.zeros_like(c)
    v = np.zeros_like(c)
    xs = np.stack([x, x])
    t0 = time.perf_counter()
    steps = 0
    while steps < 1 or time.perf_counter() - t0 < budget_s:
        t = steps + 1
        y = olin.adapted_linear_pm(xs, w, None, ut, c.reshape(N, r), 1e-3, 1, t, 0, 0, "bf16")
        g = oadam.projected_grad(oloss.mse(y[0], tgt), oloss.mse(y[1], tgt), 1e-3)
        c, m, v, _ = oadam.zo_adam(c, m, v, g, orng.gauss_range(1, t, 0, 0, N * r), oadam.adam_scalars(1e-4, t))
        steps += 1
    dt = time.perf_counter() - t0
    return {"value": round(steps / dt, 4), "unit": "ZO steps/s", "kind": "oracle",
            "sample": f"{steps} full steps ({T} tokens per half, d={K}, r={r}), {dt:.1f} s"}


# ------------------------------------------------------------------ headline: single adapted linear
def bench_single_linear(args, dev):
    import torch

    import synth
    from paper_2607_01125_amd import zoact as Z

    T, K, N, r = 8192, 4096, 4096, 32
    eps, lr, seed = 1e-3, 1e-4, 1
    x, q = synth.planted_lowrank(T, K, seed=0)
    xb = torch.from_numpy(synth.bf16_round(x)).to(dev).to(torch.bfloat16)
    # both halves read this x: the step forms x W^T and P = x U once and each half adds its
    # own rank-r correction (ZOACT_SHARED_X, the same bits as giving x twice); the stacked
    # form [2][T][K] is timed beside it for reference
    x_pm = torch.cat([xb, xb], dim=0).contiguous()
    w = torch.from_numpy(synth.bf16_round(synth.normal((N, K), 0.02, 0, 2))).to(dev).to(torch.bfloat16)
    # in-subspace teacher: Y = x (W + C* Q_r^T)^T, C* ~ N(0, 0.05^2), planted directions Q_r
    cstar = torch.from_numpy(synth.normal((N, r), 0.05, 0, 4)).to(dev)
    qr = torch.from_numpy(q[:, :r].copy()).to(dev)
    tgt = (xb.float() @ (w.float() + cstar @ qr.T).T).to(torch.bfloat16).contiguous()

    # one-shot basis (Algorithm 1) on the calibration activations, timed separately
    ut = torch.empty(r, K, dtype=torch.bfloat16, device=dev)
    eigv = torch.empty(r, dtype=torch.float32, device=dev)
    ws_b = torch.empty(Z.basis_init_workspace_bytes(K, r), dtype=torch.uint8, device=dev)
    Z.basis_init(xb, r, ut, ws_b, eigvals=eigv)       # first call loads the code objects
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    Z.basis_init(xb, r, ut, ws_b, eigvals=eigv)
    torch.cuda.synchronize()
    init_ms = (time.perf_counter() - t0) * 1e3
    del ws_b

    c = torch.zeros(N * r, dtype=torch.float32, device=dev)
    arena = Z.Arena(c, torch.zeros_like(c), torch.zeros_like(c))
    layer = Z.Linear(w, K, N, r, ut, 0)
    p = torch.empty(T, r, dtype=torch.bfloat16, device=dev)
    p_pm = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev)
    loss = torch.zeros(2, dtype=torch.float32, device=dev)
    ws_l = torch.empty(Z.linear_mse_workspace_bytes(T, N), dtype=torch.uint8, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()

    ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev)
    layer.ch, layer.ch_stride = ch, N * r

    # ch holds C +/- eps Z for step ch_for[0]: each step's update also writes the next step's
    # perturbed coefficients (zoact_step_perturb: one pass over the arena instead of two
    # launches); a step whose perturbation is not there yet forms it first
    ch_for = [None]

    def zo_step(t, ev=None, shared=True):
        pert = Z.Pert(seed, t, 0, eps)
        if ch_for[0] != t:
            Z.perturb_coeffs(arena, 0, N * r, pert, ch)
        if shared:
            Z.project(xb, ut, p)
        else:
            Z.project(x_pm, ut, p_pm)
        if ev is not None:
            ev[0].record(stream)
        # both halves' forward with the regression loss summed in the GEMM epilogue (y is
        # never stored), then the fixed-order sum of the per-tile partials
        if shared:
            Z.linear_mse(layer, arena, xb, T, p, pert, tgt, loss, ws_l, flags=Z.SHARED_X)
        else:
            Z.linear_mse(layer, arena, x_pm, T, p_pm, pert, tgt, loss, ws_l)
        if ev is not None:
            ev[1].record(stream)
        Z.step_perturb(arena, loss, pert, Z.adam_desc(lr, t), Z.Pert(seed, t + 1, 0, eps), ch, status)
        ch_for[0] = t + 1

    def timed(t0, n, shared):
        evs = [(TimingEvent(), TimingEvent()) for _ in range(n)]
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for i in range(n):
            zo_step(t0 + i, evs[i], shared)
        stop.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(stop) / n, sum(a.elapsed_time(b) for a, b in evs) / n

    for t in range(1, args.warmup + 1):
        zo_step(t)
    torch.cuda.synchronize()
    ms_per_step, gemm_ms = timed(args.warmup + 1, args.steps, True)
    losses = [float(v) for v in loss.cpu().numpy()]
    # the stacked form (x given twice, base formed per half), same steps continued
    t_next = args.warmup + 1 + args.steps
    zo_step(t_next, shared=False)
    st_steps = max(args.steps, 5)
    st_ms, st_gemm_ms = timed(t_next + 1, st_steps, False)
    gemm_flops = 2 * T * N * K + 2 * (2 * T) * r * N
    st_gemm_flops = 2 * (2 * T) * N * K + 2 * (2 * T) * r * N
    assert int(status.item()) == 0, "non-finite projected gradient"
    return {
        "workload": "single adapted linear, bf16, d_in=d_out=4096, r=32, 8192 tokens per half, planted low-rank x "
                    "(projection + fused ± forward with the MSE in its epilogue + ZO-Adam whose pass also forms the "
                    "next step's C±εZ)",
        "stacked": {"steps_per_s": round(1e3 / st_ms, 3), "ms_per_step": round(st_ms, 4),
                    "gemm_us": round(st_gemm_ms * 1e3, 1),
                    "gemm_tflops": round(st_gemm_flops / (st_gemm_ms * 1e-3) / 1e12, 1),
                    "gemm_frac": round(st_gemm_flops / (st_gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
                    "note": "x given for both halves (M=16384 stacked rows): the form the survey's cfg2 counts "
                            "(2MNK + 2MrN = 554.0 GFLOP per launch)"},
        "shared_x": {"steps_per_s": round(1e3 / ms_per_step, 3), "ms_per_step": round(ms_per_step, 4),
                     "gemm_us": round(gemm_ms * 1e3, 1),
                     "gemm_tflops": round(gemm_flops / (gemm_ms * 1e-3) / 1e12, 1),
                     "note": "both halves read one x: x W^T and x U formed once (279.2 GFLOP per launch); "
                             "reported beside the stacked form, never as it"},
        "basis_init_ms": round(init_ms, 1),
        "losses": losses,
    }


# ------------------------------------------------------------------ adapted linear at the 8B layer shapes
def bench_linear_shapes(dev, reps=10):
    """perturbed coefficients + projection + fused +/- GEMM per Llama-3-8B layer shape,
    M = 8192 stacked rows, r = 32."""
    import torch

    import synth
    from paper_2607_01125_amd import zoact as Z

    T, r = 4096, 32
    shapes = [("qkv", 4096, 6144, 0), ("o", 4096, 4096, 0), ("gate|up", 4096, 28672, Z.EPI_SWIGLU),
              ("down", 14336, 4096, 0)]
    out = {}
    # int4: the in-register INT4 GEMM; int4_dequant: one dequantisation pass into a bf16
    # buffer, then the bf16 schedule (what the decoder runs), the pass inside the timed call
    for mode in ("bf16", "int4", "int4_dequant"):
        res, tot_flop, tot_s = {}, 0.0, 0.0
        for name, K, N, flags in shapes:
            x = synth.device_normal((2 * T, K), 1.0, 9, K, device=dev, dtype=torch.bfloat16)
            w = synth.device_normal((N, K), 0.02, 9, N, K, device=dev, dtype=torch.bfloat16)
            ut = synth.device_normal((r, K), 1.0 / math.sqrt(K), 9, r, K, device=dev, dtype=torch.bfloat16)
            packed = scales = None
            if mode == "int4":
                packed, scales = synth.device_quantize_int4_g128(w)
                layer = Z.Linear(packed, K, N, r, ut, 0, w_scales=scales)
                del w
            elif mode == "int4_dequant":
                packed, scales = synth.device_quantize_int4_g128(w)
                layer = Z.Linear(w, K, N, r, ut, 0)      # w: the buffer the pass fills
            else:
                layer = Z.Linear(w, K, N, r, ut, 0)
            c = torch.zeros(N * r, dtype=torch.float32 if mode == "bf16" else torch.bfloat16, device=dev)
            arena = Z.Arena(c, torch.zeros(N * r, device=dev), torch.zeros(N * r, device=dev))
            p = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev)
            y = torch.empty(2 * T, N // 2 if flags else N, dtype=torch.bfloat16, device=dev)
            pert = Z.Pert(3, 1, 0, 1e-3)
            # C +/- eps Z formed once per step for the layer's slice, as the model step does
            ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev)
            layer.ch, layer.ch_stride = ch, N * r

            def call():
                if mode == "int4_dequant":
                    Z.dequant_int4(packed, scales, layer.w)
                Z.perturb_coeffs(arena, 0, N * r, pert, ch)
                Z.project(x, ut, p)
                Z.linear_fwd_pm(layer, arena, x, T, p, y, pert, flags=flags)

            call()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                call()
            e1.record()
            torch.cuda.synchronize()
            sec = e0.elapsed_time(e1) / reps * 1e-3
            M = 2 * T
            flop = 2 * M * N * K + 2 * M * K * r + 2 * M * r * N
            res[name] = {"M": M, "N": N, "K": K, "us": round(sec * 1e6, 1), "tflops": round(flop / sec / 1e12, 1)}
            tot_flop += flop
            tot_s += sec
            del x, layer, arena, p, y, ch, packed, scales
            torch.cuda.empty_cache()
        mean = tot_flop / tot_s / 1e12
        out[mode] = {"shapes": res, "flop_weighted_tflops": round(mean, 1),
                     "frac_of_bf16_peak": round(mean / PEAK_BF16_TFLOPS, 4)}
        log(f"8B shapes {mode}: {mean:.1f} TFLOP/s")
    out["ranks_o_shape_bf16"] = bench_ranks(dev, reps)
    return out


def bench_ranks(dev, reps, ranks=(1, 8, 32, 64, 128, 256)):
    """perturbed coefficients + projection + fused GEMM of the o-projection shape
    (M = 8192 stacked rows, N = K = 4096) across adapter ranks."""
    import torch

    import synth
    from paper_2607_01125_amd import zoact as Z

    T, K, N = 4096, 4096, 4096
    x = synth.device_normal((2 * T, K), 1.0, 9, K, device=dev, dtype=torch.bfloat16)
    w = synth.device_normal((N, K), 0.02, 9, N, K, device=dev, dtype=torch.bfloat16)
    y = torch.empty(2 * T, N, dtype=torch.bfloat16, device=dev)
    res = {}
    for r in ranks:
        ut = synth.device_normal((r, K), 1.0 / math.sqrt(K), 9, r, K, device=dev, dtype=torch.bfloat16)
        layer = Z.Linear(w, K, N, r, ut, 0)
        arena = Z.Arena(torch.zeros(N * r, device=dev), torch.zeros(N * r, device=dev), torch.zeros(N * r, device=dev))
        p = torch.empty(2 * T, r, dtype=torch.bfloat16, device=dev)
        ch = torch.empty(2 * N * r, dtype=torch.bfloat16, device=dev)
        layer.ch, layer.ch_stride = ch, N * r
        pert = Z.Pert(3, 1, 0, 1e-3)

        def call():
            Z.perturb_coeffs(arena, 0, N * r, pert, ch)
            Z.project(x, ut, p)
            Z.linear_fwd_pm(layer, arena, x, T, p, y, pert)

        call()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            call()
        e1.record()
        torch.cuda.synchronize()
        sec = e0.elapsed_time(e1) / reps * 1e-3
        M = 2 * T
        flop = 2 * M * N * K + 2 * M * K * r + 2 * M * r * N
        res[str(r)] = {"us": round(sec * 1e6, 1), "tflops": round(flop / sec / 1e12, 1)}
        del ut, layer, arena, p, ch
    log("ranks (o shape): " + ", ".join(f"r={k} {v['tflops']}" for k, v in res.items()))
    return res


# ------------------------------------------------------------------ full models
# Algorithm 1 over a model: adaptive subspace iteration to a residual of 1e-4 of
# theta_1, estimated every 8 iterations, at most 64 (sites that miss it are reported)
BASIS_TOL = 1e-4


def basis_opts():
    from paper_2607_01125_amd import zoact as Z
    return Z.EigOpts(0, 64, 0x5EED, BASIS_TOL, 1, 8)


def summarise_basis_report(rep: dict) -> dict:
    """Per-model convergence summary of Decoder.basis_report: worst residual, smallest gap
    theta_r / theta_{r+1}, iterations, sites that missed the bound; and the same per site kind."""
    import numpy as np

    def summ(vals):
        res = [v["resid"] for v in vals]
        gap = [v["gap"] for v in vals]
        its = [v["iters"] for v in vals]
        return {"sites": len(vals), "not_converged": sum(not v["converged"] for v in vals),
                "resid_max": float(f"{max(res):.3g}"), "resid_median": float(f"{float(np.median(res)):.3g}"),
                "gap_min": round(min(gap), 5), "gap_median": round(float(np.median(gap)), 5),
                "iters_min": min(its), "iters_median": int(np.median(its)), "iters_max": max(its)}
    kinds = sorted({site for (_, site) in rep})
    out = summ(list(rep.values()))
    out["tol"] = BASIS_TOL
    out["by_site"] = {k: summ([v for (l, site), v in rep.items() if site == k]) for k in kinds}
    return out


def model_step_flops(shape, B, S):
    """Algorithmic FLOPs of one +/- step: both halves' linears, LM head, causal attention,
    projection (once per adapted site) and correction."""
    M = 2 * B * S
    d, dkv, ff, V, r, L = shape.d_model, shape.n_kv_heads * shape.head_dim, shape.d_ff, shape.vocab, shape.rank, \
        shape.n_layers
    if shape.family == "llama":
        nk = [(d, d), (dkv, d), (dkv, d), (d, d), (ff, d), (ff, d), (d, ff)]
        width = {"q": d, "k": dkv, "v": dkv, "o": d, "gate": ff, "up": ff, "down": d}
        site_in = {"attn": d, "o": d, "mlp": d, "down": ff}
        sites = {"attn": {"q", "k", "v"}, "o": {"o"}, "mlp": {"gate", "up"}, "down": {"down"}}
    else:
        nk = [(d, d), (d, d), (d, d), (d, d), (ff, d), (d, ff)]
        width = {"q": d, "v": d, "o": d, "fc1": ff, "fc2": d}
        site_in = {"attn": d, "o": d, "mlp": d, "down": ff}
        sites = {"attn": {"q", "v"}, "o": {"o"}, "mlp": {"fc1"}, "down": {"fc2"}}
    ad = set(shape.adapted)
    lin = 2 * M * sum(n * k for n, k in nk) * L
    head = 2 * M * d * V
    attn = 4 * B * shape.n_heads * S * S * shape.head_dim * L          # both halves, QK^T and PV, causal half
    proj = 2 * M * r * sum(site_in[s] for s, ps in sites.items() if ps & ad) * L
    corr = 2 * M * r * sum(width[p] for p in ad) * L
    return lin + head + attn + proj + corr


class LaunchTimer:
    """Decoder.linear_hook that brackets every linear launch with fence-free HIP events on
    the current stream, recording the launch's shape; the events are preallocated so the
    timed loop creates none."""

    def __init__(self, n_max):
        self.pool = [(TimingEvent(), TimingEvent()) for _ in range(n_max)]
        self.used = []
        self.on = False

    def __call__(self, stage, lin, T, flags):
        if not self.on:
            return
        import torch

        stream = torch.cuda.current_stream()
        if stage == "pre":
            if len(self.used) >= len(self.pool):
                raise RuntimeError("LaunchTimer: event pool exhausted")
            ev = self.pool[len(self.used)]
            ev[0].record(stream)
            plain = lin.plain[1] - lin.plain[0] if lin.r else 0
            self.used.append((ev, lin.d_in, lin.d_out, lin.r, T, flags, plain))
        else:
            self.used[-1][0][1].record(stream)

    def summary(self):
        """Adapted-linear launches (r > 0): algorithmic FLOPs and durations, per shape and in total."""
        import paper_2607_01125_amd.zoact as Z

        shapes, n, tot_f, tot_s = {}, 0, 0.0, 0.0
        for (e0, e1), K, N, r, T, flags, plain in self.used:
            if r == 0:
                continue
            shared = bool(flags & Z.SHARED_X)
            n_out = N // 2 if flags & Z.EPI_SWIGLU else N
            # the correction covers the adapted features only (a plain range has none)
            f = (2 * T * N * K if shared else 2 * (2 * T) * N * K) + 2 * (2 * T) * r * (N - plain)
            sec = e0.elapsed_time(e1) * 1e-3
            key = (f"{2 * T}x{N}x{K}" + (" shared" if shared else "") + (" swiglu" if flags & Z.EPI_SWIGLU else "")
                   + (f" ({plain} features plain)" if plain else ""))
            d = shapes.setdefault(key, {"launches": 0, "flop": f, "s": 0.0, "out_features": n_out})
            d["launches"] += 1
            d["s"] += sec
            n += 1
            tot_f += f
            tot_s += sec
        per = {k: {"launches": v["launches"], "mean_us": round(v["s"] / v["launches"] * 1e6, 1),
                   "gflop_per_launch": round(v["flop"] / 1e9, 2),
                   "tflops": round(v["flop"] * v["launches"] / v["s"] / 1e12, 1)} for k, v in shapes.items()}
        return n, tot_f, tot_s, per


def bench_model(dev, which, warmup=2, steps=5, extras=True, roofline=False, workload=HEADLINE):
    import torch

    import synth
    from paper_2607_01125_amd import model as gm
    from paper_2607_01125_amd import zoact as Z

    if which in ("llama_bf16", "llama_int4"):
        shape, B, S, CB, CS, lr = synth.LLAMA3_8B, 16, 256, 16, 256, 5e-5
    else:
        shape, B, S, CB, CS, lr = synth.OPT_13B, 8, 512, 32, 512, 2.5e-5
    t0 = time.perf_counter()
    W = synth.device_model_weights(shape, 0, torch.bfloat16, device=dev)
    mode = "bf16"
    if which == "llama_int4":
        mode = "int4"
        for l in range(shape.n_layers):
            for n in ("wq", "wk", "wv", "wo", "wg", "wu", "wd"):
                W[l][n] = synth.device_quantize_int4_g128(W[l][n])
    g = gm.Decoder(shape, W, mode, device=dev)
    del W
    torch.cuda.empty_cache()
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t0
    calib = torch.from_numpy(synth.uniform_tokens(CB, CS, shape.vocab, 0, 1)).to(dev)
    tok = torch.from_numpy(synth.uniform_tokens(B, S, shape.vocab, 0, 2)).to(dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    g.basis_init(calib, basis_opts(), report=True)
    torch.cuda.synchronize()
    init_s = time.perf_counter() - t0
    basis = summarise_basis_report(g.basis_report)
    log(f"{which}: basis {basis['sites']} sites, {basis['not_converged']} above tol, resid max "
        f"{basis['resid_max']}, gap min {basis['gap_min']}, iterations {basis['iters_min']}-{basis['iters_max']}")
    timer = None
    if roofline:
        timer = LaunchTimer(steps * (6 * shape.n_layers + 8))   # at most 5 linears per layer (OPT: q|v, k, o, fc1, fc2)
        g.linear_hook = timer
    for _ in range(warmup):
        g.step(tok, 1, 1e-3, lr)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if timer is not None:
        timer.on = True
    e0.record()
    for _ in range(steps):
        g.step(tok, 1, 1e-3, lr)
    e1.record()
    torch.cuda.synchronize()
    if timer is not None:
        timer.on = False
        g.linear_hook = None
    ms = e0.elapsed_time(e1) / steps
    flops = model_step_flops(shape, B, S)
    rec = {"steps_per_s": round(1e3 / ms, 3), "ms_per_step": round(ms, 2),
           "model_tflops": round(flops / (ms * 1e-3) / 1e12, 1), "step_tflop": round(flops / 1e12, 2),
           "basis_init_s": round(init_s, 3), "basis": basis, "calibration_tokens": CB * CS, "tokens_per_half": B * S,
           "rank": shape.rank, "k": g.k, "losses": [float(v) for v in g.loss_pm.cpu().numpy()],
           "status": int(g.status.item()), "setup_s": round(setup_s, 1)}
    if timer is not None:
        n, tot_f, tot_s, per = timer.summary()
        achieved = tot_f / tot_s / 1e12
        sites = "q|k|v, o, gate|up with SwiGLU, down" if which != "opt_bf16" else "q|v, o, fc1 with ReLU, fc2"
        rec["roofline"] = {
            "kernel": f"{DOMINANT_KERNEL} (fused ± adapted GEMM) over the {n} adapted-linear launches of the "
                      f"{steps} timed steps ({n // steps} per step: {sites} per layer; "
                      f"M = {2 * B * S} stacked rows, r = {shape.rank})",
            "bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic_record(DOMINANT_KERNEL, workload, DOMINANT_SOURCES),
            "flops_per_launch": round(tot_f / n), "mean_launch_us": round(tot_s / n * 1e6, 1),
            "launches": n, "per_shape": per,
            "gemm_share_of_step": round(tot_s / (ms * 1e-3 * steps), 4)}
    if extras and which in ("llama_bf16", "llama_int4"):
        # ZO-Adam over the model's arena (HBM-bound): 24 B per coefficient (fp32 C), 20 (bf16 C)
        pert = Z.Pert(1, 99, 0, 1e-3)
        adam = Z.adam_desc(lr, 99)
        Z.step(g.arena, g.loss_pm, pert, adam, g.status)
        torch.cuda.synchronize()
        reps = 20
        e0.record()
        for _ in range(reps):
            Z.step(g.arena, g.loss_pm, pert, adam, g.status)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        per = 20 if g.c_bf16 else 24
        gbs = g.k * per / (us * 1e-6) / 1e9
        rec["adam"] = {"coefficients": g.k, "bytes_per_coefficient": per, "us": round(us, 1),
                       "achieved_GBps": round(gbs, 1), "peak_GBps": PEAK_HBM_GBS,
                       "frac": round(gbs / PEAK_HBM_GBS, 4)}
        # the update pass that also writes the next step's C +/- eps Z (the step's own form):
        # 24 (20) bytes of the update plus 4 bytes of perturbed coefficients per coefficient
        ch = torch.empty(2 * g.k, dtype=torch.bfloat16, device=dev)
        nxt = Z.Pert(1, 100, 0, 1e-3)
        Z.step_perturb(g.arena, g.loss_pm, pert, adam, nxt, ch, g.status)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            Z.step_perturb(g.arena, g.loss_pm, pert, adam, nxt, ch, g.status)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        gbs = g.k * (per + 4) / (us * 1e-6) / 1e9
        rec["adam_perturb"] = {"bytes_per_coefficient": per + 4, "us": round(us, 1), "achieved_GBps": round(gbs, 1),
                               "frac": round(gbs / PEAK_HBM_GBS, 4)}
        # the coefficient pass alone (C +/- eps Z over the arena): 4 (2) + 4 bytes per coefficient
        Z.perturb_coeffs(g.arena, 0, g.k, nxt, ch)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            Z.perturb_coeffs(g.arena, 0, g.k, nxt, ch)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        pb = (2 if g.c_bf16 else 4) + 4
        gbs = g.k * pb / (us * 1e-6) / 1e9
        rec["perturb"] = {"bytes_per_coefficient": pb, "us": round(us, 1), "achieved_GBps": round(gbs, 1),
                          "frac": round(gbs / PEAK_HBM_GBS, 4)}
        del ch
        # Algorithm 2's one-sided form with q = 8 queries: L and L_1..L_8 in five stacked
        # forwards, then the update that regenerates eight Gaussians per coefficient
        q = 8
        g.step_q(tok, 1, 1e-3, lr, q)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(2):
            g.step_q(tok, 1, 1e-3, lr, q)
        e1.record()
        torch.cuda.synchronize()
        qms = e0.elapsed_time(e1) / 2
        losses = torch.full((q + 1,), 2.0, dtype=torch.float32, device=dev)
        Z.step_q(g.arena, losses, q, 1, 99, 1e-3, adam, g.status)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            Z.step_q(g.arena, losses, q, 1, 99, 1e-3, adam, g.status)
        e1.record()
        torch.cuda.synchronize()
        qus = e0.elapsed_time(e1) / reps * 1e3
        rec["one_sided_q8"] = {"ms_per_step": round(qms, 2), "forwards_per_step": (q + 2) // 2,
                               "steps_per_s": round(1e3 / qms, 3), "update_us": round(qus, 1),
                               "update_GBps": round(g.k * per / (qus * 1e-6) / 1e9, 1)}
    del g
    torch.cuda.empty_cache()
    log(f"{which}: {rec['steps_per_s']} steps/s, {rec['model_tflops']} TFLOP/s, init {rec['basis_init_s']} s"
        + (f", GEMM {rec['roofline']['achieved']} TFLOP/s" if "roofline" in rec else "")
        + (f", one-sided q=8 {rec['one_sided_q8']['ms_per_step']} ms/step" if "one_sided_q8" in rec else ""))
    return rec


def bench_tiny(dev, steps=20):
    """The tiny fp32 model (2 layers, d = 128, r = 8 on q and v, 4 x 64 tokens): its 20 ZO
    steps after the basis from 4 x 64 calibration tokens (launch-bound; steps/s only)."""
    import torch

    import synth
    from paper_2607_01125_amd import model as gm

    shape = synth.TINY
    g = gm.Decoder(shape, synth.model_weights(shape, 0, "fp32"), "fp32", device=dev)
    g.basis_init(torch.from_numpy(synth.uniform_tokens(4, 64, shape.vocab, 0, 1)).to(dev))
    tok = torch.from_numpy(synth.uniform_tokens(4, 64, shape.vocab, 0, 2)).to(dev)
    g.step(tok, 0, 1e-3, 1e-4)
    g.t = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.step(tok, 0, 1e-3, 1e-4)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    return {"steps": steps, "steps_per_s": round(steps / dt, 1), "ms_per_step": round(dt / steps * 1e3, 3),
            "losses_last": [float(v) for v in g.loss_pm.cpu().numpy()]}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=HEADLINE, choices=list(WORKLOADS),
                    help="the workload of the JSON line (default: the headline)")
    ap.add_argument("--quick", action="store_true", help="that workload only")
    ap.add_argument("--models", default="llama_int4,opt_bf16",
                    help="comma-separated further model runs (llama_int4, opt_bf16; empty for none)")
    ap.add_argument("--no-shapes", action="store_true", help="skip the 8B layer-shape sweep")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="also run one plain device copy of this many MiB (reference for HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (the multi-GPU path is a "
              f"design, not a build)", file=sys.stderr)
        sys.exit(2)

    import torch

    dev = torch.device("cuda:0")
    which, wtext, wconf = WORKLOADS[args.workload]
    log(f"headline: {args.workload}")
    head = bench_model(dev, which, warmup=args.warmup, steps=args.steps, extras=not args.quick, roofline=True,
                       workload=args.workload)
    ms = head["ms_per_step"]
    out = {
        "metric": METRIC,
        "value": head["steps_per_s"],
        "unit": "ZO steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (random-init weights N(0, 0.02^2), uniform random tokens, seeded)",
        "config": {"workload": wtext, **wconf, "parallelism": "single GPU"},
        "model_tflops": head["model_tflops"],
        "step_tflop": head["step_tflop"],
        "basis_init_s": head["basis_init_s"],
        "roofline": head["roofline"],
        "losses": head["losses"],
        args.workload.replace("_step", ""): {k: v for k, v in head.items() if k not in ("roofline", "losses")},
    }
    log(f"headline: {out['value']} steps/s, fused GEMM {head['roofline']['achieved']} TFLOP/s "
        f"({head['roofline']['frac']:.3f} of peak)")
    if not args.quick:
        out["single_linear_4096"] = bench_single_linear(args, dev)
        log(f"single linear: stacked {out['single_linear_4096']['stacked']['steps_per_s']} steps/s "
            f"({out['single_linear_4096']['stacked']['gemm_tflops']} TFLOP/s), shared x "
            f"{out['single_linear_4096']['shared_x']['steps_per_s']} steps/s")
        if not args.no_shapes:
            out["adapted_linear_8b_shapes"] = bench_linear_shapes(dev)
        runs = [w for w in args.models.split(",") if w]
        for w in runs:
            if w not in ("llama_int4", "opt_bf16"):
                raise SystemExit(f"unknown model run {w!r}")
        if runs:
            out["models"] = {w: bench_model(dev, w) for w in runs}
        out["tiny_fp32_20_steps"] = bench_tiny(dev)
        log(f"tiny fp32: {out['tiny_fp32_20_steps']['steps_per_s']} steps/s")
    if args.calibrate_copy_mib:
        n = args.calibrate_copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_calibration_bytes"] = n
        del src, dst
    if not args.no_cpu_baseline and args.workload == HEADLINE:
        log("cpu baseline (oracle, sampled headline step)")
        out["cpu_baseline"] = cpu_baseline_llama()
        log(f"cpu baseline: {out['cpu_baseline']['seconds_per_step']} s per step (extrapolated)")
        if not args.quick:
            out["cpu_baseline_single_linear"] = cpu_baseline_single(8192, 4096, 4096, 32)
            import synth
            out["cpu_baseline_basis_init"] = cpu_baseline_basis(synth.LLAMA3_8B, 16 * 256)
            log(f"cpu baseline, basis init: {out['cpu_baseline_basis_init']['value']} s (extrapolated)")
            for w in out.get("models", {}):
                out["models"][w]["cpu_baseline"] = cpu_baseline_model(w)
                if w == "opt_bf16":
                    out["models"][w]["cpu_baseline_basis_init"] = cpu_baseline_basis(synth.OPT_13B, 32 * 512)
                log(f"cpu baseline, {w}: {out['models'][w]['cpu_baseline']['seconds_per_step']} s per step "
                    f"(extrapolated)")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
