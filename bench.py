#!/usr/bin/env python3
"""Benchmark of the RFF linear-attention hot path on one MI355X.

One step = one forward + one backward pass of causal nonstationary RFF linear
attention (feature maps formed on chip, chunked causal forward, backward for
Q, K, V, both frequency matrices and tau) over one batch of seeded synthetic
inputs already resident in HBM.  Default workload: B=2, H=16, N=8192, d=64,
m=128 frequencies per matrix (d'=256), bf16 inputs, fp32 states and gradients.

Prints ONE JSON line: throughput (tokens/s, tokens = B*N per step), the
roofline position of the dominant kernel (HIP events on its launch stream,
algorithmic bytes or flops per launch), and the float64 CPU oracle timed on a
bounded sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tokens/s, causal RFF linear-attn fwd+bwd (N=8192,d=64); % MFMA/HBM roofline"
PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
PEAK_FP32_TFLOPS = 157.3
KERNEL_FILES = {"fwd_state": "flex_fwd.hip", "fwd_sweep": "flex_fwd.hip", "scan": "flex_fwd.hip",
                "bwd_prepass": "flex_bwd.hip", "bwd_dq": "flex_bwd_dq.hip", "bwd_dkv": "flex_bwd.hip",
                "bwd_reduce": "flex_bwd.hip", "decode_step": "flex_decode.hip",
                "awd_fwd": "flex_awd.hip", "awd_bwd_k": "flex_awd.hip",
                "awd_wgrad": "flex_awd.hip"}


# transcendental VALU rate: 256 CUs x 4 SIMDs x 16 lanes per clock at quarter
# rate x 2.4 GHz
PEAK_TRANS_PER_S = 256 * 4 * 16 / 4 * 2.4e9


def _trans_per_row(wl, with_psi=False):
    """Transcendentals of one feature-map evaluation of one row: sin and cos of
    every frequency (stationary), plus cos P2 (nonstationary; plus sin P2 where
    the backward needs dphi/dP2), plus one exp for the norm factor."""
    if wl.variant == "nonstationary":
        return (4 if with_psi else 3) * wl.m + 1
    return 2 * wl.m + 1


def kernel_work(wl, kernel):
    """Algorithmic (bytes, flops, transcendentals) of one launch of a kernel
    class for a workload: the inputs it must read and the outputs it must write
    once, the contractions of the method it performs, and the feature maps it
    must evaluate (no recomputation, intra-chunk masking overhead, state
    hand-off or padding counted)."""
    T = wl.B * wl.H * wl.N                        # (b,h,token) rows
    bio = 2 if wl.io == "bf16" else 4
    d, dv, dp = wl.d, wl.dv, 2 * wl.m
    meff = 2 * wl.m if wl.variant == "nonstationary" else wl.m
    proj = 2 * d * meff                           # one row onto all frequencies
    state = 2 * dp * (dv + 1)                     # one row into / out of the state
    tr, trp = _trans_per_row(wl), _trans_per_row(wl, True)
    if kernel == "fwd_state":
        return T * 2 * d * bio, T * (proj + state), T * tr
    if kernel == "fwd_sweep":
        if not wl.causal:   # reads Q, writes O and den; phi(Q) and the readout
            return T * (2 * d * bio + 4), T * (proj + state), T * tr
        return T * (4 * d * bio + 4), T * (2 * proj + 2 * state), T * 2 * tr
    if kernel == "bwd_prepass":
        return T * (5 * d * bio + 4 + 8), T * (2 * proj + 2 * state), T * 2 * tr
    if kernel == "bwd_dq":
        # with the forward's states (as the bench runs it) the sweep also does
        # the pre-pass's query-side work: reads Q, K, V, dO, O and den; writes
        # dQ, 1/den and delta; adds the R' local state to its contractions
        return T * (5 * d * bio + 4 + 8 + 4 * d), T * (2 * state + 2 * proj), T * trp
    if kernel == "bwd_dkv":
        # reads Q, K, V, dO, 1/den and delta; writes dK, dV; dphi(K), dV, dK, dW' and R'
        return T * (4 * d * bio + 8 + 8 * d), T * (3 * state + 2 * proj), T * trp
    return 0, 0, 0


def step_work(wl, backward):
    """Algorithmic (bytes, flops, transcendentals) of one step: each input read
    and each output written once, the method's contractions (forward:
    projections of Q and K and the state / readout contractions; backward: the
    four state contractions and the chain rule's two products per projection),
    and each row's feature map once per pass (twice with the backward)."""
    BH, N, d, dv, m = wl.B * wl.H, wl.N, wl.d, wl.dv, wl.m
    bio = 2 if wl.io == "bf16" else 4
    nmat = 2 if wl.variant == "nonstationary" else 1
    meff = nmat * m
    dp = 2 * m
    wbytes = nmat * wl.H * m * d * 4
    b = BH * (3 * N * d * bio + N * dv * bio) + wbytes
    f = BH * (4 * N * d * meff + 4 * N * dp * (dv + 1))
    t = BH * 2 * N * _trans_per_row(wl)
    if backward:
        b += BH * (4 * N * d * bio + N * dv * bio + 4 * N + 3 * N * d * 4) + 2 * wbytes + BH * 4 * N
        f += BH * (8 * N * dp * (dv + 1) + 8 * N * meff * d)
        t += BH * 2 * N * _trans_per_row(wl)
    return b, f, t


def roofs_of(wl, work):
    """Roof times (s) of (bytes, flops, transcendentals) on MI355X: HBM 8 TB/s,
    dense MFMA at the io dtype's peak, transcendentals at the quarter-rate
    VALU's 9.8e12/s."""
    b, f, t = work
    peak_f = (PEAK_BF16_TFLOPS if wl.io == "bf16" else PEAK_FP32_TFLOPS) * 1e12
    return {"hbm": b / (PEAK_HBM_GBS * 1e9), "mfma": f / peak_f, "trans": t / PEAK_TRANS_PER_S}


def roofline_entry(wl, work, seconds):
    """Position of `work` done in `seconds` against its binding roof (the
    largest of the three roof times)."""
    b, f, t = work
    roofs = roofs_of(wl, work)
    bound = max(roofs, key=roofs.get)
    if bound == "hbm":
        e = {"bound": "hbm", "achieved": b / seconds / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    elif bound == "mfma":
        e = {"bound": "mfma", "achieved": f / seconds / 1e12,
             "peak": PEAK_BF16_TFLOPS if wl.io == "bf16" else PEAK_FP32_TFLOPS, "unit": "TFLOP/s"}
    else:
        e = {"bound": "alu", "achieved": t / seconds / 1e12, "peak": PEAK_TRANS_PER_S / 1e12,
             "unit": "Ttranscendental/s"}
    e["frac"] = e["achieved"] / e["peak"]
    e["roof_us"] = {k: round(v * 1e6, 2) for k, v in roofs.items()}
    e["frac_per_roof"] = {k: round(v / seconds, 4) for k, v in roofs.items()}
    return e


def copy_bandwidth_gbs(nbytes=1 << 30, reps=10):
    """Read + write bandwidth of a plain device copy of nbytes (the practical
    HBM ceiling), timed with events on the current stream."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    gbs = 2 * nbytes / (e0.elapsed_time(e1) / reps * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return gbs


def source_hash(kernel):
    src = os.path.join(ROOT, "paper_2606_27748_amd", "csrc")
    name = KERNEL_FILES.get(kernel, "flex_fwd.hip")
    files = [name, "flex_common.hpp", "flex_stage.hpp"]
    if name.startswith("flex_bwd"):
        files.append("flex_bwd_common.hpp")
    h = hashlib.sha256()
    for p in files:
        with open(os.path.join(src, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_from_profiles(workload, kernel):
    """HBM bytes per launch measured with rocprofv3 counters (committed under
    profiles/), or None when absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", f"counters_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_hash") != source_hash(kernel):
        return None
    # the class's counted bytes per step (one launch per step, or the frequency
    # groups' launches together), like `achieved`
    return rec.get("hbm_bytes_per_step", rec.get("hbm_bytes_per_launch"))


def host_facts():
    """The host the CPU baseline ran on: logical CPUs, CPU model, NumPy and its
    BLAS, and the BLAS thread pools (threadpoolctl)."""
    import numpy as np
    facts = {"os_cpu_count": os.cpu_count(), "numpy": np.__version__}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    facts["cpu_model"] = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        facts["affinity_cpus"] = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        pass
    try:
        from threadpoolctl import threadpool_info
        facts["blas"] = [{"api": i.get("internal_api"), "version": i.get("version"),
                          "threads": i.get("num_threads")} for i in threadpool_info()]
    except Exception as e:   # noqa: BLE001 (the facts are informative only)
        facts["blas"] = f"unavailable: {e}"
    return facts


def cpu_baseline(wl, slices, seed_offset=0):
    """Time the float64 oracle (forward + backward) on `slices` (b,h) slices of
    the workload at full sequence length; scale to the whole batch.  `cores`
    is the threads the run kept busy on average (CPU time over wall time)."""
    import oracle
    import workloads as W
    sub = wl.scaled(B=1, H=slices)
    x = W.generate(sub)
    t0, c0 = time.perf_counter(), time.process_time()
    oracle.linattn_bwd(x.f64("Q"), x.f64("K"), x.f64("V"), x.W1, x.W2, x.tau, x.f64("dO"),
                       wl.variant, wl.causal)
    t1, c1 = time.perf_counter(), time.process_time()
    per_step = (t1 - t0) * (wl.B * wl.H) / slices
    return {"value": wl.B * wl.N / per_step, "unit": "tokens/s",
            "cores": max(1, int(round((c1 - c0) / (t1 - t0)))), "kind": "oracle",
            "cpu_s_per_wall_s": round((c1 - c0) / (t1 - t0), 2),
            "sample": f"{slices} of {wl.B * wl.H} (b,h) slices at N={wl.N}, forward+backward in "
                      f"float64 ({t1 - t0:.1f} s), scaled by {wl.B * wl.H}/{slices}",
            "host": host_facts()}


FLUSH_BYTES = 512 << 20   # twice the 256 MB last-level cache


def step_stats(step, reps, cold):
    """Per-step time (ms) of `reps` single steps, each bracketed by events on
    the current stream; cold: a 512 MiB buffer is written before each step so
    that no input of the step is left in the last-level cache.  Returns the
    median and the 10th / 90th percentiles."""
    import torch
    flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda:0") if cold else None
    times = []
    for _ in range(reps):
        if cold:
            flush.fill_(1.0)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        step()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    times.sort()

    def pct(q):
        return times[min(len(times) - 1, int(round(q * (len(times) - 1))))]
    return {"median_ms": pct(0.5), "p10_ms": pct(0.1), "p90_ms": pct(0.9), "reps": reps}


def measure(wl, steps, warmup, want_cpu, cpu_slices, profile_only=False):
    """Time `steps` steps of a workload (after `warmup`), events on the dominant
    kernel class; returns the JSON record (None with profile_only)."""
    import torch
    import workloads as W
    import paper_2606_27748_amd as F

    dev = "cuda:0"
    x = W.generate(wl, with_grad=True)

    def dev_t(a):
        import numpy as np
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    Q, K, V, dO = dev_t(x.Q), dev_t(x.K), dev_t(x.V), dev_t(x.dO)
    W1, W2, tau = dev_t(x.W1), dev_t(x.W2), dev_t(x.tau)
    desc = F.make_desc(wl.B, wl.H, wl.N, wl.d, wl.m, wl.variant, wl.causal, wl.io)
    O = torch.empty_like(V)
    den = torch.empty(wl.B, wl.H, wl.N, dtype=torch.float32, device=dev)
    f32 = torch.float32
    backward = wl.backward
    if backward:
        try:
            F.workspace_size(desc, F.FLEX_PASS_BWD)
        except F.FlexError:
            backward = False        # shape without a backward: forward only, said in the record
    grads = dict(dQ=torch.empty(Q.shape, dtype=f32, device=dev), dK=torch.empty(K.shape, dtype=f32, device=dev),
                 dV=torch.empty(V.shape, dtype=f32, device=dev),
                 dW1=torch.empty(W1.shape, dtype=f32, device=dev),
                 dW2=None if W2 is None else torch.empty(W2.shape, dtype=f32, device=dev),
                 dtau=torch.empty(tau.shape, dtype=f32, device=dev))
    ws_f = torch.empty(F.workspace_size(desc, F.FLEX_PASS_FWD) + 256, dtype=torch.uint8, device=dev)
    ws_b = (torch.empty(F.workspace_size(desc, F.FLEX_PASS_BWD) + 256, dtype=torch.uint8, device=dev)
            if backward else None)

    def step():
        F.flex_linattn_fwd(desc, Q, K, V, W1, W2, tau, O=O, den=den, ws=ws_f)
        if backward:
            F.flex_linattn_bwd(desc, Q, K, V, W1, W2, tau, O, den, dO, ws=ws_b, fwd_ws=ws_f, **grads)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    if profile_only:
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        return None

    # which kernel class dominates (outside the timed region)
    classes = ["fwd_state", "fwd_sweep", "scan"] + (
        ["bwd_prepass", "bwd_dq", "bwd_dkv", "bwd_reduce"] if backward else [])
    share = {}
    for k in classes:
        F.flex_timing_enable(k)
        for _ in range(3):
            step()
        torch.cuda.synchronize()
        ms, n = F.flex_timing_read()
        share[k] = ms / 3
    dominant = max(share, key=share.get)

    # timed region: exactly K steps, synchronized on both sides, events on the dominant kernel
    F.flex_timing_enable(dominant)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    k_ms, k_n = F.flex_timing_read()
    F.flex_timing_enable("none")
    ms_step = (t1 - t0) * 1e3 / steps
    tokens = wl.B * wl.N
    value = tokens / (ms_step * 1e-3)

    # the same loop with no timing events, for comparison (outside the contract's region)
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms_step_noev = (time.perf_counter() - t2) * 1e3 / steps

    # the step captured once in a HIP graph and replayed K times (outside the
    # contract's region: the library launches only kernels on the caller's
    # stream, so the whole step captures)
    try:
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            step()
        for _ in range(3):
            graph.replay()
        torch.cuda.synchronize()
        t3 = time.perf_counter()
        for _ in range(steps):
            graph.replay()
        torch.cuda.synchronize()
        ms_step_graph = (time.perf_counter() - t3) * 1e3 / steps
    except RuntimeError as e:
        ms_step_graph = f"capture failed: {e}"

    # the class's time per step (several launches when the shape runs as
    # frequency groups) against its algorithmic work per step
    per_step = max(k_n // steps, 1)
    avg_s = (k_ms / steps) * 1e-3
    kwl = wl if backward == wl.backward else wl.scaled(backward=False)
    roof = roofline_entry(wl, kernel_work(kwl, dominant), avg_s)
    roof["traffic"] = traffic_from_profiles(wl.name, dominant)
    roof["kernel"] = dominant
    roof["kernel_ms"] = avg_s * 1e3
    roof["launches_per_step"] = per_step
    roof["kernel_share"] = {k: round(v / sum(share.values()), 4) for k, v in share.items()}
    copy_gbs = copy_bandwidth_gbs()
    if roof["bound"] == "hbm":
        roof["copy_gbs"] = copy_gbs
        roof["frac_vs_copy"] = roof["achieved"] / copy_gbs
    # the whole step against its own binding roof
    step_roof = roofline_entry(wl, step_work(wl, backward), ms_step * 1e-3)
    step_roof["copy_gbs"] = copy_gbs
    if step_roof["bound"] == "hbm":
        step_roof["frac_vs_copy"] = step_roof["achieved"] / copy_gbs
    roof["step"] = step_roof

    out = {"metric": METRIC, "value": value, "unit": "tokens/s", "n_gpus": 1, "steps": steps,
           "warmup": warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16" if wl.io == "bf16" else "f32", "data": "synthetic",
           "config": {"workload": wl.name, "B": wl.B, "H": wl.H, "N": wl.N, "d": wl.d, "m": wl.m,
                      "variant": wl.variant, "causal": wl.causal,
                      "pass": "fwd+bwd" if backward else "fwd", "parallelism": "single-gpu"},
           "roofline": roof}
    out["step_timing"] = {"warm": step_stats(step, 20, False), "cold": step_stats(step, 20, True),
                          "flush_bytes": FLUSH_BYTES, "ms_per_step_no_events": ms_step_noev,
                          "ms_per_step_graph": ms_step_graph,
                          "note": "value and ms_per_step: the contract's K back-to-back steps, warm "
                                  "(a step's inputs, outputs and workspaces stay in the 256 MB "
                                  "last-level cache where they fit); cold: single steps with a "
                                  "512 MiB buffer written before each, so no input is cached"}
    cold = out["step_timing"]["cold"]["median_ms"]
    out["value_cold"] = tokens / (cold * 1e-3)
    if wl.backward and not backward:
        out["config"]["note"] = "backward not built for this shape; forward only"
    if want_cpu:
        out["cpu_baseline"] = cpu_baseline(wl, min(cpu_slices, wl.B * wl.H))
    else:
        out["cpu_baseline"] = None
    return out


def device_bytes(wl):
    """Device memory a call needs: inputs, outputs and both workspaces."""
    import paper_2606_27748_amd as F
    rows = wl.B * wl.H * wl.N
    bio = 2 if wl.io == "bf16" else 4
    nmat = 2 if wl.variant == "nonstationary" else 1
    desc = F.make_desc(wl.B, wl.H, wl.N, wl.d, wl.m, wl.variant, wl.causal, wl.io)
    tensors = rows * wl.d * bio * 4 + rows * 4 + nmat * wl.H * wl.m * wl.d * 4   # Q, K, V, O, den, W
    ws = F.workspace_size(desc, F.FLEX_PASS_FWD)
    if wl.backward:
        tensors += rows * wl.d * bio + rows * wl.d * 4 * 3 + nmat * wl.H * wl.m * wl.d * 4  # dO, dQ/dK/dV, dW
        ws += F.workspace_size(desc, F.FLEX_PASS_BWD)
    return tensors, ws


def run_sweep(steps, warmup):
    """Time per step and device memory against the sequence length N (fixed B*H,
    causal nonstationary d=64, m=128, forward and forward+backward) and against
    the number of frequencies m (d=64, N=8192): the paper's cost-versus-length
    and cost-versus-n comparisons, on synthetic inputs, for this implementation
    only."""
    import workloads as W
    base = W.WORKLOADS["headline_causal_train_d64"]
    cases = []
    for N in (1024, 2048, 4096, 8192, 16384, 32768):
        for bwd in (False, True):
            cases.append(("N", base.scaled(name=f"sweep_N{N}_{'fwdbwd' if bwd else 'fwd'}", N=N, backward=bwd)))
    for variant in ("nonstationary", "stationary"):
        for m in (64, 128, 192, 256):
            cases.append(("m", base.scaled(name=f"sweep_m{m}_{variant[:4]}", m=m, variant=variant)))
    for axis, wl in cases:
        rec = measure(wl, steps, warmup, False, 0)
        tensors, ws = device_bytes(wl)
        print(json.dumps({"axis": axis, "workload": wl.name, "N": wl.N, "m": wl.m, "variant": wl.variant,
                          "pass": rec["config"]["pass"], "ms_per_step": rec["ms_per_step"],
                          "tokens_per_s": rec["value"], "device_bytes": tensors + ws,
                          "workspace_bytes": ws, "dominant_kernel": rec["roofline"]["kernel"],
                          "roofline_frac": rec["roofline"]["frac"]}), flush=True)


AWD_CLASSES = ("feature_map", "awd_fwd", "awd_bwd_k", "awd_wgrad")


def awd_kernel_work(wl, kernel):
    """Algorithmic (bytes, MFMA flops, transcendentals) of one launch of a
    distillation kernel class: the inputs it must read and the outputs it must
    write once, and the method's contractions (the logit tile Q K^T, the kernel
    tile phi phi^T, and G phi for each side), excluding the recomputation of the
    S and A tiles in the gradient passes."""
    S, N, d, F = wl.B * wl.H, wl.N, wl.d, 2 * wl.m
    bio = 2 if wl.io == "bf16" else 4
    pairs = S * N * N
    if kernel == "awd_fwd":
        # reads Q, K, phi(Q), phi(K), z; writes (lse, 1/den) per query and dphi(Q);
        # the logit and kernel tiles and G phi(K); exp, log and a reciprocal per pair
        return (S * (2 * N * d * bio + 2 * N * F * bio + F * 4 + N * 8 + N * F * bio),
                pairs * (2 * d + 4 * F), 3 * pairs)
    if kernel == "awd_bwd_k":
        # reads both sides' rows and features and the statistics; writes dphi (io dtype)
        return (S * (2 * N * d * bio + 2 * N * F * bio + N * 8 + N * F * bio), pairs * 2 * F, 2 * pairs)
    if kernel == "awd_wgrad":
        m_eff = wl.m * (2 if wl.variant == "nonstationary" else 1)
        rows = 2 * S * N
        return rows * (d * bio + F * bio), rows * (2 * d * m_eff) * 2, rows * (3 if m_eff > wl.m else 2) * wl.m
    if kernel == "feature_map":
        m_eff = wl.m * (2 if wl.variant == "nonstationary" else 1)
        rows = 2 * S * N   # the rows of Q and of K, mapped in one launch
        return rows * (d * bio + F * bio), rows * 2 * d * m_eff, rows * (3 if m_eff > wl.m else 2) * wl.m
    return 0, 0, 0


def run_awd(steps, warmup, want_cpu, cpu_batches=32):
    """One distillation step = flex_awd_loss with gradients (the loss of every
    (b,h) slice and dW1, dW2, dtau) on the distillation workload, inputs
    resident in HBM."""
    import torch
    import workloads as W
    import paper_2606_27748_amd as F
    wl = W.AWD_WORKLOADS[W.AWD_HEADLINE]
    dev = "cuda:0"
    x = W.generate_awd(wl)

    def dev_t(a):
        import numpy as np
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    Q, K, W1, W2, tau = dev_t(x.Q), dev_t(x.K), dev_t(x.W1), dev_t(x.W2), dev_t(x.tau)
    desc = F.make_desc(wl.B, wl.H, wl.N, wl.d, wl.m, wl.variant, False, wl.io)
    f32 = torch.float32
    outs = dict(loss=torch.empty(wl.B, wl.H, dtype=f32, device=dev),
                dW1=torch.empty(W1.shape, dtype=f32, device=dev),
                dW2=None if W2 is None else torch.empty(W2.shape, dtype=f32, device=dev),
                dtau=torch.empty(tau.shape, dtype=f32, device=dev))
    ws = torch.empty(F.workspace_size(desc, F.FLEX_PASS_AWD) + 256, dtype=torch.uint8, device=dev)

    def step():
        F.flex_awd_loss(desc, Q, K, W1, W2, tau, ws=ws, **outs)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    share = {}
    for k in AWD_CLASSES:
        F.flex_timing_enable(k)
        for _ in range(3):
            step()
        torch.cuda.synchronize()
        ms, n = F.flex_timing_read()
        share[k] = ms / 3
    dominant = max(share, key=share.get)
    F.flex_timing_enable(dominant)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    k_ms, k_n = F.flex_timing_read()
    F.flex_timing_enable("none")
    ms_step = (t1 - t0) * 1e3 / steps
    avg_s = (k_ms / steps) * 1e-3
    kb, kf, kt = awd_kernel_work(wl, dominant)
    peak_f = PEAK_BF16_TFLOPS if wl.io == "bf16" else PEAK_FP32_TFLOPS
    roofs = {"hbm": kb / (PEAK_HBM_GBS * 1e9), "mfma": kf / (peak_f * 1e12), "alu": kt / PEAK_TRANS_PER_S}
    bound = max(roofs, key=roofs.get)
    if bound == "hbm":
        roof = {"bound": "hbm", "achieved": kb / avg_s / 1e9, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    elif bound == "mfma":
        roof = {"bound": "mfma", "achieved": kf / avg_s / 1e12, "peak": peak_f, "unit": "TFLOP/s"}
    else:
        roof = {"bound": "alu", "achieved": kt / avg_s / 1e12, "peak": PEAK_TRANS_PER_S / 1e12,
                "unit": "Ttranscendental/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = traffic_from_profiles(wl.name, dominant)
    roof["kernel"] = dominant
    roof["kernel_ms"] = avg_s * 1e3
    roof["launches_per_step"] = max(k_n // steps, 1)
    roof["roof_us"] = {k: round(v * 1e6, 2) for k, v in roofs.items()}
    roof["kernel_share"] = {k: round(v / sum(share.values()), 4) for k, v in share.items()}
    out = {"metric": "tokens/s, attention-weight distillation loss + dW1/dW2/dtau (N=512, d=64)",
           "value": wl.B * wl.N / (ms_step * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": steps,
           "warmup": warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16" if wl.io == "bf16" else "f32", "data": "synthetic",
           "config": {"workload": wl.name, "B": wl.B, "H": wl.H, "N": wl.N, "d": wl.d, "m": wl.m,
                      "variant": wl.variant, "causal": False, "pass": "loss+grad"},
           "roofline": roof,
           "step_timing": {"warm": step_stats(step, 20, False), "cold": step_stats(step, 20, True),
                           "flush_bytes": FLUSH_BYTES}}
    if want_cpu:
        import oracle
        sub = wl.scaled(B=cpu_batches)
        xs = W.generate_awd(sub)
        c0, p0 = time.perf_counter(), time.process_time()
        oracle.awd_grads(xs.f64("Q"), xs.f64("K"), xs.W1, xs.W2, xs.tau, wl.variant)
        c1, p1 = time.perf_counter(), time.process_time()
        per_step = (c1 - c0) * wl.B / cpu_batches
        out["cpu_baseline"] = {"value": wl.B * wl.N / per_step, "unit": "tokens/s",
                               "cores": max(1, int(round((p1 - p0) / (c1 - c0)))), "kind": "oracle",
                               "sample": f"{cpu_batches} of {wl.B} batches (all {wl.H} heads, N={wl.N}): loss "
                                         f"and gradient in float64 ({c1 - c0:.1f} s), scaled by {wl.B}/{cpu_batches}"}
    else:
        out["cpu_baseline"] = None
    return out


def run_decode(steps, warmup, B=256, H=16, d=64, m=128):
    """Decode steps of the causal nonstationary attention for a batch of B
    sequences (one new token each per step) against the resident fp32 state.
    The state read-modify-write bounds the step: its bytes, the token rows and
    the frequencies (read once per step) are the algorithmic traffic."""
    import torch
    import paper_2606_27748_amd as F
    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(7)
    s = d ** -0.25
    q = (torch.randn(B, H, d, device=dev, generator=g) * s).to(torch.bfloat16)
    k = (torch.randn(B, H, d, device=dev, generator=g) * s).to(torch.bfloat16)
    v = (torch.randn(B, H, d, device=dev, generator=g) * s).to(torch.bfloat16)
    W1 = torch.randn(H, m, d, device=dev, generator=g)
    W2 = torch.randn(H, m, d, device=dev, generator=g)
    tau = torch.full((H,), math.log(2.0), device=dev)
    desc = F.make_desc(B, H, 1, d, m, "nonstationary", True, "bf16")
    state = F.decode_state(desc)
    o = torch.empty(B, H, d, dtype=torch.bfloat16, device=dev)
    den = torch.empty(B, H, device=dev)
    for _ in range(warmup):
        F.flex_decode_step(desc, q, k, v, W1, W2, tau, state, o, den)
    torch.cuda.synchronize()
    F.flex_timing_enable("decode_step")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        F.flex_decode_step(desc, q, k, v, W1, W2, tau, state, o, den)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    k_ms, _ = F.flex_timing_read()
    F.flex_timing_enable("none")
    ms = (t1 - t0) * 1e3 / steps
    kernel_ms = k_ms / steps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # the practical ceiling: a device copy of the state (read + write), same timing
    dst = torch.empty_like(state)
    for _ in range(3):
        dst.copy_(state)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        dst.copy_(state)
    e1.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * state.numel() * 4 / (e0.elapsed_time(e1) / steps * 1e-3) / 1e9
    del dst
    nbytes = B * H * (2 * m) * (d + 1) * 4 * 2 + B * H * d * 2 * 4 + B * H * 4 + 2 * H * m * d * 4
    workload = f"decode_nonstationary_B{B}_H{H}_d{d}_m{m}"
    return {"metric": "tokens/s, causal RFF linear-attn decode step", "value": B / (ms * 1e-3),
            "unit": "tokens/s", "n_gpus": 1, "steps": steps, "warmup": warmup, "ms_per_step": ms,
            "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": workload, "B": B, "H": H, "d": d, "m": m,
                       "state_bytes": B * H * 2 * m * (d + 1) * 4},
            "roofline": {"bound": "hbm", "achieved": nbytes / (kernel_ms * 1e-3) / 1e9,
                         "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": nbytes / (kernel_ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                         "traffic": traffic_from_profiles(workload, "decode_step"),
                         "kernel": "decode_step", "kernel_ms": kernel_ms,
                         "algorithmic_bytes": nbytes, "state_copy_gbs": copy_gbs}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="headline_causal_train_d64")
    ap.add_argument("--all-configs", action="store_true",
                    help="one JSON line per configured workload (no CPU baseline)")
    ap.add_argument("--awd", action="store_true",
                    help="attention-weight distillation loss and its kernel-parameter gradient")
    ap.add_argument("--decode", action="store_true",
                    help="recurrent decode step (one token per sequence against the running state)")
    ap.add_argument("--decode-batch", type=int, default=256,
                    help="sequences per decode step (the default state, 272 MB, exceeds the 256 MB last-level cache)")
    ap.add_argument("--sweep", action="store_true",
                    help="scaling sweep: time and device memory against N and against m (JSON lines)")
    ap.add_argument("--cpu-slices", type=int, default=32)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--profile-only", action="store_true",
                    help="run warmup + steps only (for rocprofv3); no JSON")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run plain 1 GiB device copies (calibrates rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda:0")   # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": src.numel() * 4, "launches": 3}))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} is not supported "
              "(the path is built for one GPU; it has no multi-GPU sharding)", file=sys.stderr)
        sys.exit(2)

    import workloads as W
    if args.sweep:
        run_sweep(args.steps, args.warmup)
        return
    if args.awd:
        print(json.dumps(run_awd(args.steps, args.warmup, not args.no_cpu)), flush=True)
        return
    if args.decode:
        print(json.dumps(run_decode(args.steps, args.warmup, B=args.decode_batch)), flush=True)
        return
    if args.all_configs:
        for name, wl in W.WORKLOADS.items():
            print(json.dumps(measure(wl, args.steps, args.warmup, False, 0)), flush=True)
        return
    wl = W.WORKLOADS[args.workload]
    out = measure(wl, args.steps, args.warmup, not args.no_cpu, args.cpu_slices, args.profile_only)
    if out is not None:
        print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
