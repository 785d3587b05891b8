"""Benchmark of the reproducible fp32 operators on one MI355X.

One step is the backward pass of a Llama-shaped linear layer, the largest
workload that fits one GPU: dX = dY.W^T (8192 x 4096, K = 14336) and
dW = X^T.dY (4096 x 14336, K = 8192 tokens), 1.924 TFLOP per step, X ~ N(0,1),
dY ~ N(0,1e-2), W ~ N(0,0.02^2), canonical 64-block k order.  Both products are
timed with HIP events on the stream they run on, each kernel separately.  A
fixed-duration clock ramp of the same products runs before the counted warmup
(the matrix-core clocks need tens of milliseconds of sustained work to reach
their steady state).  The same run times the other workloads (the 2048^3 GEMM,
the row reductions and elementwise operators at their model shapes, the
model-shaped pipelines) as secondary figures, and the CPU oracle on a bounded
sample of the headline workload (cpu_baseline).  Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--launch mfma:0]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP32_VECTOR_PEAK_TFLOPS = 157.3  # MI355X published dense fp32 peak (vector and matrix alike)
HBM_PEAK_GBPS = 8000.0           # MI355X published HBM3E bandwidth
METRIC = "bit-exact reproducible fp32 GEMM GFLOP/s (% fp32 vector peak); softmax/LN GB/s"


def parse_launch(spec, repops):
    if spec in (None, "", "auto"):
        return None
    kind, _, idx = spec.partition(":")
    kinds = {"simple": repops.LAUNCH_GEMM_SIMPLE, "tiled": repops.LAUNCH_GEMM_TILED,
             "mfma": repops.LAUNCH_GEMM_MFMA}
    if kind == "simple":
        return repops.Launch(kinds[kind])
    return repops.Launch(kinds[kind], (int(idx or 0),))


COUNTERS_MD = os.path.join(ROOT, "profiles", "llama_linear_backward_hbm_counters.md")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2502_19405_amd", "csrc", f)
                  for f in ("gemm_mfma.hip", "gemm_store.h", "repops_internal.h", "api.cpp")]


def kernel_source_sha256():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(launch_spec, product):
    """HBM bytes per launch of one headline product ("dX" or "dW") from the
    committed rocprofv3 counter summary, or None when the summary does not
    cover this kernel as it now stands (other launch, changed sources)."""
    if launch_spec not in ("auto", "mfma:0") or not os.path.exists(COUNTERS_MD):
        return None
    fields = {}
    for line in open(COUNTERS_MD):
        key, eq, val = line.partition(" = ")
        if eq:
            fields[key.strip()] = val.strip()
    if fields.get("kernel_source_sha256") != kernel_source_sha256():
        return None
    val = fields.get(f"traffic_bytes_per_launch_{product}")
    return float(val) if val else None


# Shortest timed region of a secondary workload (see event_time_ms); 0 keeps
# every workload at exactly its given number of calls (the counter passes
# count dispatches per workload).
MIN_TIMED_MS = 2.0
# Calls the last event_time_ms / graph_time_ms made (warmup and capture
# included); _rate reports it, so a kernel trace of the run can be split into
# workloads call for call.
_LAUNCHED = [0]
_RAMPED = [0]  # untimed clock-ramp calls since the last _rate


def event_time_ms(fn, reps, warmup=2, min_total_ms=None):
    """Average duration of fn() over reps launches, HIP events on the current
    stream (the stream the library launches on).  Calls of a few microseconds
    are timed over enough launches to fill min_total_ms (MIN_TIMED_MS unless
    given; the first, shorter timing then serves as further warmup), so that
    the average is steady."""
    import torch
    if min_total_ms is None:
        min_total_ms = MIN_TIMED_MS
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()

    def timed(n):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for _ in range(n):
            fn()
        stop.record()
        stop.synchronize()
        return start.elapsed_time(stop)
    total = timed(reps)
    _LAUNCHED[0] = warmup + reps
    if total < min_total_ms:
        reps = min(int(reps * min_total_ms / max(total, 1e-3)) + 1, 20000)
        total = timed(reps)
        _LAUNCHED[0] += reps
    return total / reps


class ClockSampler:
    """Samples the GPU's current shader clock (the starred level of the
    kernel driver's pp_dpm_sclk table) every few milliseconds in a background
    thread; median() is None where the table is not readable or ambiguous."""

    def __init__(self, period_s=0.01):
        import glob
        import threading
        paths = glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk")
        self.path = paths[0] if len(paths) == 1 else None
        self.samples, self.period, self._stop = [], period_s, threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)

    def _read(self):
        try:
            for line in open(self.path):
                if line.strip().endswith("*"):
                    return int(line.split(":")[1].strip().rstrip("*").strip().lower().rstrip("mhz"))
        except (OSError, ValueError, IndexError):
            return None
        return None

    def _run(self):
        while not self._stop.is_set():
            v = self._read()
            if v:
                self.samples.append(v)
            self._stop.wait(self.period)

    def __enter__(self):
        if self.path:
            self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self.path:
            self._thread.join()

    def median(self):
        s = sorted(self.samples[len(self.samples) // 4:])  # past the first quarter
        return s[len(s) // 2] if s else None


def clock_ramp(fn, ms=150.0):
    """Repeat fn for a fixed wall-clock duration (untimed) so that a
    matrix-core workload is timed at steady clocks; the calls are counted into
    the next _rate figure."""
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < ms:
        fn()
        torch.cuda.synchronize()
        _RAMPED[0] += 1


GRAPHS = True  # False (--no-graphs): no graph-replayed figures


def graph_time_ms(fn, calls=20, reps=10):
    """Average duration of fn() with `calls` of them captured in one HIP graph
    and the graph replayed `reps` times: the kernels' own time without host
    launch gaps (none of the library's calls allocates or clears memory, so
    they capture as they run).  None when GRAPHS is off."""
    import torch
    if not GRAPHS:
        return None
    fn()
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(calls):
            fn()
    graph.replay()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(reps):
        graph.replay()
    stop.record()
    stop.synchronize()
    _LAUNCHED[0] = 2 + calls * (1 + reps)
    return start.elapsed_time(stop) / (calls * reps)


def _timed_rows(fn, total_rows, target_s):
    """Run fn(rows) on a growing row count until it takes about target_s (or
    covers every row); returns (rows, seconds) of the last run."""
    rows = 1
    while True:
        t0 = time.perf_counter()
        fn(rows)
        dt = time.perf_counter() - t0
        if dt > target_s / 8 or rows >= total_rows:
            break
        rows = min(total_rows, rows * 4)
    if dt < target_s and rows < total_rows:
        rows = int(min(total_rows, max(rows, rows * target_s / max(dt, 1e-3))))
        t0 = time.perf_counter()
        fn(rows)
        dt = time.perf_counter() - t0
    return rows, dt


def cpu_baseline(d, target_s=12.0):
    """The oracle, as it stands, on bounded samples: the headline's dX product
    on leading rows of dY with every host thread, and single-threaded the
    whole 256^3 GEMM and leading rows of the 2048^3 GEMM."""
    import numpy as np
    import oracle
    from paper_2502_19405_amd import inputs

    threads = oracle.default_threads()
    dY, W = d["dY"], d["W"]
    n, k = W.shape[0], W.shape[1]
    rows, dt = _timed_rows(
        lambda r: oracle.matmul(np.ascontiguousarray(dY[:r]), W, trans_b=True, nthreads=threads),
        dY.shape[0], target_s)
    gflops = rows * 2.0 * n * k / dt / 1e9
    out = {"value": round(gflops, 3), "unit": "GFLOP/s", "cores": threads, "kind": "oracle",
           "sample": f"first {rows} of {dY.shape[0]} rows of dX = dY.W^T ({n} columns, K = {k}), "
                     f"{dt:.2f} s wall on {threads} threads"}
    one = {}
    c1 = inputs.gemm256_softmax256()
    t0 = time.perf_counter()
    oracle.matmul(c1["A"], c1["B"], nthreads=1)
    dt1 = time.perf_counter() - t0
    one["gemm256"] = {"s": round(dt1, 3), "GFLOP/s": round(2 * 256 ** 3 / dt1 / 1e9, 3),
                      "sample": "whole 256^3 GEMM"}
    c2 = inputs.gemm2048_bias()
    r2, dt2 = _timed_rows(lambda r: oracle.matmul(np.ascontiguousarray(c2["A"][:r]), c2["B"],
                                                  c2["bias"], nthreads=1), 2048, 4.0)
    one["gemm2048_bias"] = {"s": round(dt2, 3), "GFLOP/s": round(r2 * 2 * 2048 ** 2 / dt2 / 1e9, 3),
                            "sample": f"first {r2} of 2048 output rows"}
    out["single_thread"] = one
    return out


def _graph_rate(ms, nbytes=None, flops=None):
    """The same figures for graph-replayed calls, keys prefixed graph_ (none
    without a measurement)."""
    if ms is None:
        return {}
    return {"graph_" + k: v for k, v in _rate(ms, nbytes, flops).items()}


def _rate(ms, nbytes=None, flops=None):
    out = {"ms": round(ms, 4), "launches": _LAUNCHED[0]}
    if _RAMPED[0]:
        out["ramp_launches"] = _RAMPED[0]
        _RAMPED[0] = 0
    if nbytes is not None:
        gbps = nbytes / ms / 1e6
        out.update({"GB/s": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)})
    if flops is not None:
        tf = flops / ms / 1e9
        out.update({"TFLOP/s": round(tf, 2), "frac_peak": round(tf / FP32_VECTOR_PEAK_TFLOPS, 4)})
    return out


def secondary(repops, steps, streaming_only=False, headline=None):
    """The other workloads, each timed with HIP events after warmup:
    row reductions and elementwise ops in GB/s of algorithmic bytes (each
    element read once and written once; causal softmax reads only the
    unmasked part), GEMM-shaped steps and the model-shaped pipelines in
    TFLOP/s of 2*M*N*K.  streaming_only keeps the bandwidth-bound operators
    and the two copies, every call launched eagerly on one stream (no graph
    replays, no GEMMs): the set the HBM byte counters are taken over.
    headline: the headline's device tensors (X, dY, dW), reused for one
    data-parallel rank's share of the dW product."""
    import numpy as np
    import torch
    from paper_2502_19405_amd import inputs, pipelines

    out = {}
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(a).to(dev)  # noqa: E731
    g = inputs.rng(4)

    # 256^3 GEMM and 256 x 256 softmax (launch-bound sizes)
    d = {} if streaming_only else inputs.gemm256_softmax256()
    if not streaming_only:
        A, B, S = t(d["A"]), t(d["B"]), t(d["S"])
        C, P = torch.empty_like(A), torch.empty_like(S)
        out["gemm_256"] = _rate(event_time_ms(lambda: repops.matmul(A, B, out=C), steps * 5),
                                flops=2 * 256 ** 3)
        out["gemm_256"].update(_graph_rate(graph_time_ms(lambda: repops.matmul(A, B, out=C)),
                                           flops=2 * 256 ** 3))
        sm = lambda: repops.softmax_rows(S, out=P)  # noqa: E731
        out["softmax_256x256"] = _rate(event_time_ms(sm, steps * 5), nbytes=8 * 256 * 256)
        out["softmax_256x256"].update(_graph_rate(graph_time_ms(sm), nbytes=8 * 256 * 256))

    # 2048^3 GEMM + bias (A, B ~ U(-1,1), bias ~ U(-0.1,0.1))
    if not streaming_only:
        c2 = inputs.gemm2048_bias()
        A2, B2, bias2 = t(c2["A"]), t(c2["B"]), t(c2["bias"])
        C2 = torch.empty((2048, 2048), device=dev)
        clock_ramp(lambda: repops.matmul(A2, B2, bias2, out=C2))
        out["gemm2048_bias"] = _rate(
            event_time_ms(lambda: repops.matmul(A2, B2, bias2, out=C2), steps * 5, warmup=20),
            flops=2 * 2048 ** 3)
        del A2, B2, bias2, C2

    # causal softmax, Llama attention scores: 4 x 32 heads x 1024 rows of 1024
    T, rows = 1024, 4 * 32 * 1024
    S = t(inputs.normal(g, (rows, T), var=4.0))
    P = torch.empty_like(S)
    ms = event_time_ms(lambda: repops.softmax_rows(S, causal_period=T, out=P), steps)
    out["softmax_causal_131072x1024"] = _rate(ms, nbytes=4 * (rows // T) * (T * (T + 1) // 2 + T * T))
    ms = event_time_ms(lambda: repops.softmax_rows(S, out=P), steps)
    out["softmax_dense_131072x1024"] = _rate(ms, nbytes=4 * rows * T * 2)
    ms = event_time_ms(lambda: repops.exp(S, out=P), steps)
    out["exp_131072x1024"] = _rate(ms, nbytes=4 * rows * T * 2)
    # 4096-wide rows (one row per workgroup, split over waves)
    S4 = S.view(-1)[:4096 * 4096].view(4096, 4096)
    P4 = P.view(-1)[:4096 * 4096].view(4096, 4096)
    ms = event_time_ms(lambda: repops.softmax_rows(S4, out=P4), steps)
    out["softmax_4096x4096"] = _rate(ms, nbytes=4 * S4.numel() * 2)
    # softmax backward on the same scores: reads Y and dY (unmasked part when
    # causal), writes dX everywhere
    Yp = repops.softmax_rows(S, causal_period=T)
    dP = t(inputs.normal(g, (rows, T), var=1e-4))
    ms = event_time_ms(lambda: repops.softmax_backward_rows(Yp, dP, causal_period=T, out=P), steps)
    out["softmax_backward_causal_131072x1024"] = _rate(
        ms, nbytes=4 * (rows // T) * (2 * T * (T + 1) // 2 + T * T))
    ms = event_time_ms(lambda: repops.softmax_backward_rows(Yp, dP, out=P), steps)
    out["softmax_backward_dense_131072x1024"] = _rate(ms, nbytes=4 * rows * T * 3)
    Y4 = Yp.view(-1)[:4096 * 4096].view(4096, 4096)
    dP4 = dP.view(-1)[:4096 * 4096].view(4096, 4096)
    P4 = P.view(-1)[:4096 * 4096].view(4096, 4096)
    ms = event_time_ms(lambda: repops.softmax_backward_rows(Y4, dP4, out=P4), steps)
    out["softmax_backward_4096x4096"] = _rate(ms, nbytes=4 * Y4.numel() * 3)
    del S, P, Yp, dP

    d = inputs.distilbert_mlp()
    gam, bet = t(d["gamma"]), t(d["beta"])
    for name, shape in (("layernorm_4096x768", (4096, 768)), ("layernorm_65536x768", (65536, 768))):
        Z = t(inputs.normal(g, shape, var=0.5))
        Y = torch.empty_like(Z)
        ms = event_time_ms(lambda: repops.layernorm_rows(Z, gam, bet, out=Y), steps)
        out[name] = _rate(ms, nbytes=4 * Z.numel() * 2)
        if shape[0] == 4096 and not streaming_only:  # launch-bound: also without launch gaps
            out[name].update(_graph_rate(
                graph_time_ms(lambda: repops.layernorm_rows(Z, gam, bet, out=Y)),
                nbytes=4 * Z.numel() * 2))
    # LayerNorm backward: reads X and dY, writes dX (mean, rstd, gamma and the
    # [cols] parameter gradients are negligible); dgamma/dbeta included
    for name, shape in (("layernorm_backward_4096x768", (4096, 768)),
                        ("layernorm_backward_65536x768", (65536, 768))):
        Z = t(inputs.normal(g, shape, var=0.5))
        mean = torch.empty(shape[0], device=dev)
        rstd = torch.empty(shape[0], device=dev)
        repops.layernorm_rows(Z, gam, bet, mean_out=mean, rstd_out=rstd)
        dZ = t(inputs.normal(g, shape, var=1e-2))
        dX = torch.empty_like(Z)
        dg, db = torch.empty_like(gam), torch.empty_like(gam)
        ws = torch.empty(max(repops.layernorm_backward_workspace(*shape) // 4, 1), device=dev)
        call = lambda: repops.layernorm_backward_rows(  # noqa: E731
            Z, dZ, mean, rstd, gam, dx_out=dX, dgamma_out=dg, dbeta_out=db, workspace=ws)
        out[name] = _rate(event_time_ms(call, steps), nbytes=4 * Z.numel() * 3)
        if shape[0] == 4096 and not streaming_only:
            out[name].update(_graph_rate(graph_time_ms(call), nbytes=4 * Z.numel() * 3))
        del Z, dZ, dX, ws
    H = t(inputs.normal(g, (4096, 3072), var=0.31))
    G = torch.empty_like(H)
    out["gelu_4096x3072"] = _rate(event_time_ms(lambda: repops.gelu(H, out=G), steps),
                                  nbytes=4 * H.numel() * 2)
    dG = t(inputs.normal(g, (4096, 3072), var=1e-2))
    out["gelu_backward_4096x3072"] = _rate(
        event_time_ms(lambda: repops.gelu_backward(H, dG, out=G), steps), nbytes=4 * H.numel() * 3)
    out["gelu_erf_4096x3072"] = _rate(event_time_ms(lambda: repops.gelu_erf(H, out=G), steps),
                                      nbytes=4 * H.numel() * 2)
    out["gelu_erf_backward_4096x3072"] = _rate(
        event_time_ms(lambda: repops.gelu_erf_backward(H, dG, out=G), steps),
        nbytes=4 * H.numel() * 3)
    del H, G, dG
    # Adam: reads param, grad, exp_avg, exp_avg_sq and writes three of them
    # (28 B per parameter); the DistilBERT feed-forward block's 4.72 M
    # parameters, and a 64 M-parameter flat buffer
    for name, n in (("adam_4723968", 2 * 768 * 3072 + 3072 + 3 * 768),
                    ("adam_67108864", 1 << 26)):
        p = t(inputs.normal(g, (n,), var=4e-4))
        gr = t(inputs.normal(g, (n,), var=1e-4))
        m, v = torch.zeros_like(p), torch.zeros_like(p)
        ms = event_time_ms(lambda: repops.adam_step(p, gr, m, v, 1e-4, weight_decay=0.01, step=10),
                           steps)
        out[name] = _rate(ms, nbytes=28 * n)
        del p, gr, m, v

    # Llama-block operators: rotary embedding of Q (4 x 1024 tokens, 32 heads of
    # 128; 8 B per element), RMSNorm over 4096 x 4096 (forward 8 B, backward with
    # dgamma 12 B per element), SwiGLU over 4096 x 14336 (forward 12 B,
    # backward 20 B per element)
    Q = t(inputs.normal(g, (4096, 4096)))
    Qo = torch.empty_like(Q)
    inv = t((500000.0 ** (-np.arange(0, 128, 2) / 128)).astype(np.float32))
    ms = event_time_ms(lambda: repops.rope(Q, 32, 128, inv, 1024, 0, out=Qo), steps)
    out["rope_4096x32x128"] = _rate(ms, nbytes=4 * Q.numel() * 2)
    gw = t((1 + inputs.uniform(g, (4096,), -0.1, 0.1)).astype(np.float32))
    rs = torch.empty(4096, device=dev)
    ms = event_time_ms(lambda: repops.rmsnorm_rows(Q, gw, out=Qo, rstd_out=rs), steps)
    out["rmsnorm_4096x4096"] = _rate(ms, nbytes=4 * Q.numel() * 2)
    dQ = t(inputs.normal(g, (4096, 4096), var=1e-2))
    dgw = torch.empty_like(gw)
    wsr = torch.empty(max(repops.rmsnorm_backward_workspace(4096, 4096) // 4, 1), device=dev)
    ms = event_time_ms(lambda: repops.rmsnorm_backward_rows(
        Q, dQ, rs, gw, dx_out=Qo, dgamma_out=dgw, workspace=wsr), steps)
    out["rmsnorm_backward_4096x4096"] = _rate(ms, nbytes=4 * Q.numel() * 3)
    del Q, Qo, dQ, wsr
    Gt = t(inputs.normal(g, (4096 * 14336,), var=4.0))
    Ut = t(inputs.normal(g, (4096 * 14336,)))
    Yt = torch.empty_like(Gt)
    ms = event_time_ms(lambda: repops.swiglu(Gt, Ut, out=Yt), steps)
    out["swiglu_4096x14336"] = _rate(ms, nbytes=4 * Gt.numel() * 3)
    Dt = t(inputs.normal(g, (4096 * 14336,), var=1e-2))
    Et = torch.empty_like(Gt)
    ms = event_time_ms(lambda: repops.swiglu_backward(Gt, Ut, Dt, dg_out=Yt, du_out=Et), steps)
    out["swiglu_backward_4096x14336"] = _rate(ms, nbytes=4 * Gt.numel() * 5)
    del Gt, Ut, Yt, Dt, Et

    # tensor commitment (SHA-256 Merkle tree, 1 KiB leaves) of a Llama-8B
    # feed-forward weight, 4096 x 14336 fp32: bytes read once; SHA-256 is
    # integer VALU work (about 30 instructions per byte with the tree levels),
    # bound by the latency of each lane's dependent block chain
    Wc = t(inputs.normal(g, (4096, 14336), var=4e-4))
    dig = torch.empty(32, dtype=torch.uint8, device=dev)
    wsc = torch.empty(repops.commit_workspace(Wc.numel() * 4, 1024) // 4 + 1, dtype=torch.int32,
                      device=dev)
    ms = event_time_ms(lambda: repops.commit(Wc, 1024, digest=dig, workspace=wsc), steps)
    out["commit_4096x14336"] = _rate(ms, nbytes=Wc.numel() * 4)
    del Wc, wsc

    # streaming ceilings: a device-to-device copy of 512 MiB by torch's copy kernel
    src = torch.empty(1 << 27, device=dev)
    dst = torch.empty_like(src)
    ms = event_time_ms(lambda: dst.copy_(src), steps)
    out["copy_ceiling_512MiB"] = _rate(ms, nbytes=2 * 4 * src.numel())
    # The library's own elementwise kernel with no arithmetic: the streaming
    # rate the bandwidth-bound operators can reach.
    ms = event_time_ms(lambda: repops.copy(src, out=dst), steps)
    out["copy_repops_512MiB"] = _rate(ms, nbytes=2 * 4 * src.numel())
    del src, dst
    if streaming_only:
        return out

    # DistilBERT feed-forward block: 4096 tokens, 768 -> 3072 -> 768, GELU, LayerNorm
    X, W1, W2, b1, b2 = (t(d[k]) for k in ("X", "W1", "W2", "b1", "b2"))
    clock_ramp(lambda: pipelines.mlp_forward(X, W1, b1, W2, b2, gam, bet))
    ms = event_time_ms(lambda: pipelines.mlp_forward(X, W1, b1, W2, b2, gam, bet), steps)
    out["distilbert_mlp_block"] = _rate(ms, flops=2 * 2 * 4096 * 768 * 3072)
    # the same block replayed from a HIP graph: the kernels without host launch gaps
    out["distilbert_mlp_block"].update(_graph_rate(
        graph_time_ms(lambda: pipelines.mlp_forward(X, W1, b1, W2, b2, gam, bet)),
        flops=2 * 2 * 4096 * 768 * 3072))
    # one whole training step of the block: forward, every gradient, AdamW over
    # all 4.72 M parameters (six GEMMs of 2 * 4096 * 768 * 3072 flop each)
    st = pipelines.MlpTrainState(W1, b1, W2, b2, gam, bet)
    dYb = t(inputs.normal(g, (4096, 768), var=1e-4))
    sbufs = {}
    clock_ramp(lambda: pipelines.mlp_train_step(st, X, dYb, bufs=sbufs))
    ms = event_time_ms(lambda: pipelines.mlp_train_step(st, X, dYb, bufs=sbufs), steps)
    out["distilbert_mlp_train_step"] = _rate(ms, flops=6 * 2 * 4096 * 768 * 3072)
    # replayed from a HIP graph (the captured steps repeat one step's Adam
    # scalars; the kernels and their sizes are those of every step)
    out["distilbert_mlp_train_step"].update(_graph_rate(
        graph_time_ms(lambda: pipelines.mlp_train_step(st, X, dYb, bufs=sbufs), calls=5),
        flops=6 * 2 * 4096 * 768 * 3072))
    del X, W1, W2, b1, b2, st, dYb, sbufs

    # Llama attention block: 4 x 1024 tokens, d 4096, 32 heads
    d = inputs.llama_attention()
    X, Wq, Wk, Wv, Wo = (t(d[k]) for k in ("X", "Wq", "Wk", "Wv", "Wo"))
    bufs = {k: torch.empty((4096, 4096), device=dev) for k in ("Q", "K", "V", "O", "out")}
    bufs["S"] = torch.empty((4, 32, 1024, 1024), device=dev)
    bufs["P"] = torch.empty((4 * 32 * 1024, 1024), device=dev)
    fl = 4 * 2 * 4096 ** 3 + 2 * 2 * 4 * 32 * 1024 * 1024 * 128
    clock_ramp(lambda: pipelines.attention_forward(X, Wq, Wk, Wv, Wo, 4, 1024, 32, buffers=bufs))
    ms = event_time_ms(lambda: pipelines.attention_forward(X, Wq, Wk, Wv, Wo, 4, 1024, 32,
                                                           buffers=bufs), max(steps // 4, 3))
    out["llama_attention_block"] = _rate(ms, flops=fl)
    Q, K, S = bufs["Q"], bufs["K"], bufs["S"]
    ms = event_time_ms(lambda: repops.bmm_raw(4, 32, 1024, 1024, 128, Q, 1024 * 4096, 128, 4096, 0,
                                              K, 1024 * 4096, 128, 4096, 1, 0.08838835, S,
                                              32 * 1024 * 1024, 1024 * 1024, 1024), steps)
    out["bmm_qkT_4x32x1024x1024x128"] = _rate(ms, flops=2 * 4 * 32 * 1024 * 1024 * 128)
    # causal: only the scores at or below the diagonal are ever read
    out["bmm_qkT_4x32x1024x1024x128"]["causal_useful_TFLOP/s"] = round(
        2 * 4 * 32 * 128 * (1024 * 1025 // 2) / ms / 1e9, 2)
    # the causal score product: only the tiles at or below each head's diagonal
    ms = event_time_ms(lambda: repops.bmm_raw(4, 32, 1024, 1024, 128, Q, 1024 * 4096, 128, 4096, 0,
                                              K, 1024 * 4096, 128, 4096, 1, 0.08838835, S,
                                              32 * 1024 * 1024, 1024 * 1024, 1024,
                                              causal=repops.CAUSAL_OUTPUT), steps)
    out["bmm_qkT_causal"] = _rate(ms, flops=2 * 4 * 32 * 128 * (1024 * 1025 // 2))
    out["bmm_qkT_causal"]["dense_equivalent_TFLOP/s"] = round(
        2 * 4 * 32 * 1024 * 1024 * 128 / ms / 1e9, 2)
    # PV: P [4*32*1024, 1024] times V's head columns, written in place into O
    P, V, O = bufs["P"], bufs["V"], bufs["O"]
    ms = event_time_ms(lambda: repops.bmm_raw(4, 32, 1024, 128, 1024, P, 32 * 1024 * 1024,
                                              1024 * 1024, 1024, 0, V, 1024 * 4096, 128, 4096, 0,
                                              1.0, O, 1024 * 4096, 128, 4096), steps)
    out["bmm_pv_4x32x1024x128x1024"] = _rate(ms, flops=2 * 4 * 32 * 1024 * 128 * 1024)
    # causal: row i of P has i + 1 nonzero probabilities
    out["bmm_pv_4x32x1024x128x1024"]["causal_useful_TFLOP/s"] = round(
        2 * 4 * 32 * 128 * (1024 * 1025 // 2) / ms / 1e9, 2)
    # P's all-zero blocks skipped (the same bits)
    ms = event_time_ms(lambda: repops.bmm_raw(4, 32, 1024, 128, 1024, P, 32 * 1024 * 1024,
                                              1024 * 1024, 1024, 0, V, 1024 * 4096, 128, 4096, 0,
                                              1.0, O, 1024 * 4096, 128, 4096,
                                              causal=repops.CAUSAL_A), steps)
    out["bmm_pv_causal"] = _rate(ms, flops=2 * 4 * 32 * 128 * (1024 * 1025 // 2))
    out["bmm_pv_causal"]["dense_equivalent_TFLOP/s"] = round(
        2 * 4 * 32 * 1024 * 128 * 1024 / ms / 1e9, 2)
    del X, Wq, Wk, Wv, Wo, bufs, Q, K, S, P, V, O

    # the headline's two products as one grouped launch (the pipeline's path)
    if headline is not None:
        X, dY, W, gx, gw = (headline[k] for k in ("X", "dY", "W", "dX", "dW"))
        ms = event_time_ms(lambda: pipelines.linear_backward(X, dY, W, out_dx=gx, out_dw=gw), 5)
        out["llama_linear_backward_grouped"] = _rate(ms, flops=2 * 2 * 8192 * 4096 * 14336)
        del X, dY, W, gx, gw
    # one rank's share of dW under 8-way data parallelism: the headline's dW
    # product over 1024 of the 8192 tokens (the ordered cross-rank combine is
    # not built)
    if headline is not None:
        X, dY, gw = headline["X"], headline["dY"], headline["dW"]
        ms = event_time_ms(lambda: repops.matmul(X[:1024].t(), dY[:1024], out=gw), steps)
        out["llama_dW_rank_share_4096x14336x1024"] = _rate(ms, flops=2 * 4096 * 14336 * 1024)
        del X, dY, gw

    return out


def input_digests(d):
    import hashlib
    import numpy as np
    return {k: hashlib.sha256(np.ascontiguousarray(v).tobytes()).hexdigest() for k, v in d.items()}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    # The clocks take tens of milliseconds of sustained matrix-core work to
    # reach their steady state; this ramp runs before the counted warmup and
    # is not timed, so a small --warmup still measures steady clocks.
    ap.add_argument("--ramp-ms", type=float, default=300.0)
    ap.add_argument("--no-graphs", action="store_true",
                    help="leave out the graph-replayed secondary figures (counter passes)")
    ap.add_argument("--launch", default="auto",
                    help="auto | simple | tiled:I | mfma:I (auto picks mfma:0 for both products)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--streaming-only", action="store_true",
                    help="secondary workloads: only the bandwidth-bound operators and copies, "
                         "launched eagerly (for HBM byte counters)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a 256 MiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the reproducible operators shard without any "
              "exchange along their order-free dimensions, so a multi-GPU figure adds nothing "
              "here; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if args.steps < 1 or args.warmup < 0:
        print("--steps must be at least 1 and --warmup at least 0", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2502_19405_amd import inputs, repops

    repops.load()
    dev = torch.device("cuda:0")
    d = inputs.llama_linear_backward()
    digests = input_digests(d)
    T, D_IN, D_OUT = d["X"].shape[0], d["X"].shape[1], d["W"].shape[1]
    X = torch.from_numpy(d["X"]).to(dev)
    dY = torch.from_numpy(d["dY"]).to(dev)
    W = torch.from_numpy(d["W"]).to(dev)
    dX = torch.empty((T, D_IN), device=dev)
    dW = torch.empty((D_IN, D_OUT), device=dev)
    launch = parse_launch(args.launch, repops)
    Wt, Xt = W.t(), X.t()

    def prod_dx():
        repops.matmul(dY, Wt, launch=launch, out=dX)

    def prod_dw():
        repops.matmul(Xt, dY, launch=launch, out=dW)

    # untimed clock ramp: the step repeated for a fixed wall-clock duration
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ramp_steps = 0
    while (time.perf_counter() - t0) * 1e3 < args.ramp_ms:
        prod_dx()
        prod_dw()
        torch.cuda.synchronize()
        ramp_steps += 1
    ramp_ms = (time.perf_counter() - t0) * 1e3
    for _ in range(args.warmup):
        prod_dx()
        prod_dw()
    torch.cuda.synchronize()

    # timed steps: an event before dX, between the two products and after dW
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * args.steps + 1)]
    with ClockSampler() as clock:
        t0 = time.perf_counter()
        ev[0].record()
        for i in range(args.steps):
            prod_dx()
            ev[2 * i + 1].record()
            prod_dw()
            ev[2 * i + 2].record()
        torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    dx_ms = sum(ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(args.steps)) / args.steps
    dw_ms = sum(ev[2 * i + 1].elapsed_time(ev[2 * i + 2]) for i in range(args.steps)) / args.steps
    step_ms = ev[0].elapsed_time(ev[-1]) / args.steps
    flops_each = 2.0 * T * D_IN * D_OUT
    value_gflops = 2 * flops_each / (step_ms * 1e-3) / 1e9

    mfma = launch is None or launch.kind == repops.LAUNCH_GEMM_MFMA
    kernels = {}
    for name, ms, shape in (("dX", dx_ms, f"{T}x{D_IN}, K={D_OUT}, W read transposed"),
                            ("dW", dw_ms, f"{D_IN}x{D_OUT}, K={T}, X read transposed")):
        tf = flops_each / (ms * 1e-3) / 1e12
        kernels[name] = {"ms": round(ms, 4), "TFLOP/s": round(tf, 2),
                         "frac": round(tf / FP32_VECTOR_PEAK_TFLOPS, 4), "shape": shape,
                         "traffic": measured_traffic(args.launch, name)}
    dom = "dX" if dx_ms >= dw_ms else "dW"  # the kernel that takes longer
    result = {
        "metric": METRIC,
        "value": round(value_gflops, 1),
        "unit": "GFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "wall_ms_per_step": round(wall_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"llama_linear_backward: dX = dY.W^T and dW = X^T.dY, tokens {T}, "
                               f"in {D_IN}, out {D_OUT}; X ~ N(0,1), dY ~ N(0,1e-2), "
                               f"W ~ N(0,0.02^2); k_block 64, fma, left-to-right",
                   "launch": args.launch, "parallelism": "single GPU"},
        "roofline": {"bound": "mfma" if mfma else "alu", "kernel": dom,
                     "achieved": kernels[dom]["TFLOP/s"], "peak": FP32_VECTOR_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": kernels[dom]["frac"],
                     "traffic": kernels[dom]["traffic"]},
        "kernels": kernels,
        # the shader clock the chip held during the timed steps (the published
        # peak assumes 2.4 GHz) and the slower product's fraction of the peak
        # at that clock
        "sustained_clock": ({"mhz": clock.median(),
                             "frac_at_clock": round(kernels[dom]["TFLOP/s"] / (
                                 FP32_VECTOR_PEAK_TFLOPS * clock.median() / 2400.0), 4)}
                            if clock.median() else None),
        "clock_ramp": {"ms": round(ramp_ms, 1), "steps": ramp_steps},
        "inputs_sha256": digests,
    }
    if args.calibrate_copy:
        src = torch.empty(64 << 20, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        result["calibration_copy_bytes"] = src.numel() * 4
    if not args.no_secondary:
        global MIN_TIMED_MS, GRAPHS
        if args.streaming_only:
            MIN_TIMED_MS = 0.0
        GRAPHS = not args.no_graphs
        result["secondary"] = secondary(repops, 20, args.streaming_only,
                                        headline={"X": X, "dY": dY, "W": W, "dX": dX, "dW": dW})
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(d)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
