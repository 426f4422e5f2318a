"""Benchmark of the SSD layer forward on one MI355X.

One step = one ``ssd_forward`` call (every step of the block decomposition)
over one batch of seeded synthetic input already resident in HBM.  Inputs
rotate among three independent copies so that the 256 MB last-level cache
cannot serve a step from the previous one.  Prints one JSON line.

Default workload: Mamba-2-2.7B-like layer, batch 4 x seqlen 4096, 80 heads of
64, state 128, one group, chunk 256, bf16 inputs with float32 accumulation.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X published peaks
PEAK_BF16_FLOPS = 2.5e15
PEAK_F32_MFMA_FLOPS = 157.3e12
PEAK_F32_VECTOR_FLOPS = 157.3e12
PEAK_HBM_BPS = 8.0e12


def algorithmic_counts(p, nseq):
    """FLOPs (block-decomposition cost model of Section 6 with the Gram C B^T
    counted once per group, in two conventions) and compulsory HBM bytes."""
    b, T, H, P, N, G, Q = p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size
    tok = b * T
    f_full = tok * (2 * Q * N * G + H * (2 * Q * P + 4 * N * P))
    f_causal = tok * ((Q + 1) * N * G + H * ((Q + 1) * P + 4 * N * P))
    act = 2 if p.dtype == "bf16" else 4
    units = nseq if p.varlen else b
    state_bytes = units * H * P * N * 4
    byts = act * (2 * tok * H * P + tok * H + 2 * tok * G * N) + state_bytes
    if p.init_states:
        byts += state_bytes
    if p.varlen:
        byts += 4 * tok
    byts += 4 * 2 * H  # A_log, D
    return f_full, f_causal, byts


FWD_SOURCES = ("ssd_fused.hip", "ssd_device.h", "ssd_internal.h")
BWD_SOURCES = ("ssd_backward_mfma.hip", "ssd_backward.hip", "ssd_device.h", "ssd_bwd.h")


def kernel_sources_digest(sources=FWD_SOURCES):
    """Hash of the sources the measured kernels are compiled from; counter files
    record the digest they were taken at."""
    import hashlib

    h = hashlib.sha256()
    for name in sources:
        with open(os.path.join(ROOT, "paper_2405_21060_amd", "csrc", name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def dominant_kernel_name(p, general=False):
    fused = (not general and p.dtype == "bf16" and p.headdim == 64 and p.chunk_size == 256
             and p.dstate in (64, 128, 256))
    return ("k_fused_main<%d>" % p.dstate) if fused else "k_chunk_output"


def measured_traffic(workload, prefix="ssd_fused", sources=FWD_SOURCES):
    """HBM bytes per launch of the dominant kernel from the FETCH_SIZE / WRITE_SIZE
    counter runs committed under profiles/, scaled by the plain-copy calibration;
    None when there is no record for this workload or the kernels have changed
    since it was taken."""
    path = os.path.join(ROOT, "profiles", "%s_%s_traffic.json" % (prefix, workload))
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("kernel_sources_sha256_16") != kernel_sources_digest(sources):
        return None
    cal = rec["calibration"]
    k = rec["per_dispatch_kib"][rec["dominant_kernel"]]
    return int(1024 * (k["FETCH_SIZE"] * cal["fetch_factor"] + k["WRITE_SIZE"] * cal["write_factor"]))


def cpu_baseline(inp, budget_s=20.0):
    """The oracle (untuned) on the host cores, on a bounded sample of the
    workload: all tokens, a subset of heads sized to ~budget_s of CPU time."""
    import numpy as np

    import oracle

    p = inp.problem
    threads = oracle.default_threads()
    # calibrate on one head, one thread (also the 1-thread rate)
    t0 = time.perf_counter()
    oracle.forward_inputs(inp, heads=[0], nthreads=1)
    one = time.perf_counter() - t0
    nheads = int(max(1, min(p.nheads, budget_s * threads / max(one, 1e-6) / 1.5)))
    heads = list(np.linspace(0, p.nheads - 1, nheads).astype(int))
    t0 = time.perf_counter()
    oracle.forward_inputs(inp, heads=heads, nthreads=threads)
    el = time.perf_counter() - t0
    tok_per_s = p.batch * p.seqlen * (len(heads) / p.nheads) / el
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": tok_per_s, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": "all %d tokens x %d of %d heads (float64 sequential recurrence, "
                      "OpenMP over heads), %.1f s; rate scaled to all heads"
                      % (p.batch * p.seqlen, len(heads), p.nheads, el),
            "cpu_model": model,
            "one_thread_value": p.batch * p.seqlen / p.nheads / one,
            "one_thread_sample": "all %d tokens x 1 head on 1 thread, %.2f s; rate scaled to all heads"
                                 % (p.batch * p.seqlen, one)}


def decode_bench(args, torch, ssd):
    """Decode step of the 2.7B-layer shape (H80 P64 N128 G1, bf16) at batch
    --decode-batch: one step = one token for every sequence, state updated in
    place.  Bound by HBM: the state is read and written every step (at batch
    256 it is 671 MB, beyond the 256 MB last-level cache)."""
    import numpy as np

    b, H, P, N, G = args.decode_batch, 80, 64, 128, 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    g = torch.Generator(device="cpu").manual_seed(args.seed)
    x = torch.randn((b, H, P), generator=g).to(torch.bfloat16).to(dev)
    dt = (torch.rand((b, H), generator=g) * 0.1 + 1e-3).to(torch.bfloat16).to(dev)
    A_log = (torch.rand((H,), generator=g) * np.log(16.0)).to(dev)
    B = (torch.randn((b, G, N), generator=g) / np.sqrt(N)).to(torch.bfloat16).to(dev)
    C = (torch.randn((b, G, N), generator=g) / np.sqrt(N)).to(torch.bfloat16).to(dev)
    D = torch.randn((H,), generator=g).to(dev)
    state = torch.randn((b, H, P, N), generator=g).to(dev)
    y = torch.empty_like(x)
    stream = torch.cuda.current_stream(dev)
    prob = ssd.make_problem(b, 1, H, P, N, G, 256, ssd.SSD_DTYPE_BF16, 0)
    ptr = lambda t: t.data_ptr()

    def step():
        rc = ssd.ssd_decode_step(prob, ptr(x), ptr(dt), ptr(A_log), ptr(B), ptr(C), ptr(D), ptr(state),
                                 ptr(y), stream.cuda_stream)
        if rc != 0:
            raise ssd.SsdError(rc, "ssd_decode_step")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(args.steps):
        step()
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    sec = ms * 1e-3
    state_bytes = b * H * P * N * 4
    byts = 2 * state_bytes + 2 * (2 * b * H * P + b * H + 2 * b * G * N) + 8 * H
    print(json.dumps({
        "metric": "SSD decode step tokens/s (2.7B-layer shape, 1 GPU)",
        "value": b / sec, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "decode_2p7b", "batch": b, "nheads": H, "headdim": P, "dstate": N,
                   "ngroups": G},
        "roofline": {"bound": "hbm", "achieved": byts / sec / 1e9, "peak": PEAK_HBM_BPS / 1e9,
                     "unit": "GB/s", "frac": byts / sec / PEAK_HBM_BPS, "traffic": None,
                     "kernel": "k_decode_step", "algorithmic_bytes": byts},
    }), flush=True)


def block_bench(args, torch, ssd):
    """The layer with the block steps around it (ssd_forward_block) on the
    2.7B-layer workload: dt = softplus(dt_raw + bias), the layer, the gate
    y * SiLU(z) and an RMS normalisation over groups of --block-norm-group
    channels (default one head, 64).  The same call with the gate and norm left
    to the separate output pass, and the plain layer, are timed in the same run
    for comparison."""
    import os

    from paper_2405_21060_amd.inputs import WORKLOADS, make_block_inputs

    p = WORKLOADS["mamba2_2p7b"]
    bi = make_block_inputs(p, args.seed)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def act(a):
        return torch.from_numpy(a.view("int16")).view(torch.bfloat16).to(dev)

    base = bi.base
    sets = []
    for _ in range(max(1, args.copies)):
        sets.append({"x": act(base.x), "dt_raw": act(bi.dt_raw), "dt": act(base.dt), "B": act(base.B),
                     "C": act(base.C), "z": act(bi.z), "y": torch.empty_like(act(base.x))})
    A_log = torch.from_numpy(base.A_log).to(dev)
    D = torch.from_numpy(base.D).to(dev)
    bias = torch.from_numpy(bi.dt_bias).to(dev)
    w = torch.from_numpy(bi.norm_weight).to(dev)
    fin = torch.empty((p.batch, p.nheads, p.headdim, p.dstate), dtype=torch.float32, device=dev)
    prob = ssd.make_problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size,
                            ssd.SSD_DTYPE_BF16, 0)
    wsb = ssd.ssd_workspace_bytes(prob)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    ptr = lambda t: None if t is None else t.data_ptr()
    kev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, z in kev:
        a.record(stream)
        z.record(stream)

    def call(i, mode, events=None):
        c = sets[i % len(sets)]
        if mode == "layer":
            rc = ssd.ssd_forward(prob, ptr(c["x"]), ptr(c["dt"]), ptr(A_log), ptr(c["B"]), ptr(c["C"]),
                                 ptr(D), None, None, ptr(c["y"]), ptr(fin), ptr(ws), wsb, stream.cuda_stream)
        else:
            opts = ssd.make_block_opts(bias, True, 0.0, float("inf"), c["z"], w, args.block_norm_group, 1e-5)
            a = (prob, opts, ptr(c["x"]), ptr(c["dt_raw"]), ptr(A_log), ptr(c["B"]), ptr(c["C"]), ptr(D),
                 None, None, ptr(c["y"]), ptr(fin), ptr(ws), wsb, stream.cuda_stream)
            rc = ssd.ssd_forward_block_timed(*a, events[0].cuda_event, events[1].cuda_event) if events \
                else ssd.ssd_forward_block(*a)
        if rc != 0:
            raise ssd.SsdError(rc, mode)

    def timed(mode, with_events=False):
        if mode == "separate":
            ssd.ssd_set_tuning("separate_block_post", 1)
        try:
            for i in range(args.warmup):
                call(i, mode)
            torch.cuda.synchronize()
            t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0.record(stream)
            for i in range(args.steps):
                call(i, mode, kev[i] if with_events else None)
            t1.record(stream)
            torch.cuda.synchronize()
        finally:
            ssd.ssd_set_tuning("separate_block_post", 0)
        return t0.elapsed_time(t1) / args.steps

    ms = timed("block")
    timed("block", with_events=True)   # the chunk kernel's own duration (events add their own cost)
    ks = sorted(a.elapsed_time(z) for a, z in kev)
    kms = {"mean": sum(ks) / len(ks), "p10": ks[len(ks) // 10], "p50": ks[len(ks) // 2],
           "p90": ks[(9 * len(ks)) // 10]}
    ms_sep = timed("separate")
    ms_layer = timed("layer")
    _, _, byts = algorithmic_counts(p, base.nseq)
    tokens = p.batch * p.seqlen
    byts += 2 * tokens * p.nheads * p.headdim + 4 * p.nheads + 4 * p.nheads * p.headdim   # z, bias, weight
    ksec = kms["mean"] * 1e-3
    fused_norm = args.block_norm_group == p.headdim
    print(json.dumps({
        "metric": "SSD block fwd tokens/s (dt softplus + layer + SiLU gate + RMSNorm, 2.7B-layer shape, 1 GPU)",
        "value": tokens / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded; Mamba-2 layer shapes)",
        "config": {"workload": "block_mamba2_2p7b", "batch": p.batch, "seqlen": p.seqlen,
                   "nheads": p.nheads, "headdim": p.headdim, "dstate": p.dstate, "ngroups": p.ngroups,
                   "chunk_size": p.chunk_size, "norm_group_size": args.block_norm_group},
        "separate_output_pass_ms": ms_sep,
        "layer_only_ms": ms_layer,
        "roofline": {"bound": "hbm", "achieved": byts / ksec / 1e9, "peak": PEAK_HBM_BPS / 1e9,
                     "unit": "GB/s", "frac": byts / ksec / PEAK_HBM_BPS, "traffic": None,
                     "kernel": "k_fused_main<128> (dt step, gate%s fused)" % (" and norm" if fused_norm else ""),
                     "kernel_ms": kms, "algorithmic_bytes": byts},
    }), flush=True)


def backward_fast(p):
    """Whether the backward runs on its matrix-core path (bf16, headdim 64, dstate 64 or 128)."""
    return p.dtype == "bf16" and p.headdim == 64 and p.dstate in (64, 128)


def backward_counts(p):
    """Counts for the backward's dominant kernel, the chunk-gradient kernel, at
    its chunk length Qb (64 on the matrix-core path, 32 otherwise):

    * FLOPs: per head the causal (u >= t) pairs of four score-sized products
      (dy x^T and dy^T Gs over the head dimension, C^T Rs and B^T Rs^T over the
      state dimension), C B^T once per group, and three state-sized products
      per token (Gn B, Gn^T x~, h_in^T dy);
    * bytes: the backward's compulsory bytes (x, dt, B, C, dy read; dx, ddt,
      dB, dC written; A_log, D and their gradients).  The two chunk-state
      arrays the kernel also reads (h_in and Gn per chunk and head, P x N each,
      bf16 on the matrix-core path, float32 otherwise) are intermediates of
      this design, not of the problem: returned separately, never counted as
      algorithmic bytes.

    Returns (flops, algorithmic bytes, chunk-state bytes, Qb)."""
    b, T, H, P, N, G = p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups
    fast = backward_fast(p)
    Qb = 64 if fast else 32
    nC = -(-T // Qb)
    pairs = b * nC * Qb * (Qb + 1) // 2
    flops = pairs * G * N * 2 + H * (pairs * (2 * P + 2 * N) * 2 + b * T * 3 * P * N * 2)
    act = 2 if p.dtype == "bf16" else 4
    compulsory = act * (3 * b * T * H * P + 2 * b * T * H + 4 * b * T * G * N) + 4 * 4 * H
    states = 2 * b * nC * H * P * N * (2 if fast else 4)
    return flops, compulsory, states, Qb


def backward_bench(args, torch, ssd):
    """Gradients of the 2.7B-shape layer (ssd_backward): dy seeded, no initial
    state and no final-state gradient (the training case)."""
    import numpy as np

    from paper_2405_21060_amd.inputs import WORKLOADS, make_grad_inputs, make_inputs
    from paper_2405_21060_amd.device import act_to_device, to_device

    p = WORKLOADS[args.workload]
    inp = make_inputs(p, args.seed)
    dy, _ = make_grad_inputs(p, args.seed)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sets = []
    for _ in range(max(1, args.copies)):
        c = to_device(inp)
        c["dy"] = act_to_device(dy)
        c["dx"], c["ddt"] = torch.empty_like(c["x"]), torch.empty_like(c["dt"])
        c["dB"], c["dC"] = torch.empty_like(c["B"]), torch.empty_like(c["C"])
        c["dA_log"], c["dD"] = torch.empty_like(c["A_log"]), torch.empty_like(c["D"])
        sets.append(c)
    prob = ssd.make_problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size,
                            ssd.SSD_DTYPE_BF16 if p.dtype == "bf16" else ssd.SSD_DTYPE_F32, 0)
    wsb = ssd.ssd_backward_workspace_bytes(prob)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    ptr = lambda t: None if t is None else t.data_ptr()
    kev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, z in kev:
        a.record(stream)
        z.record(stream)

    starts = None
    if p.varlen:
        # packed row: the sequences' host offsets, and their initial states
        seq = inp.seq_idx.reshape(-1)
        starts = [0] + [int(v) for v in np.flatnonzero(np.diff(seq)) + 1] + [int(seq.size)]
        prob = ssd.make_problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size,
                                ssd.SSD_DTYPE_BF16 if p.dtype == "bf16" else ssd.SSD_DTYPE_F32, inp.nseq)
        wsb = ssd.ssd_backward_varlen_workspace_bytes(prob, starts)
        ws = torch.empty(wsb, dtype=torch.uint8, device=dev)

    def call(i, events=None):
        c = sets[i % len(sets)]
        if starts is not None:
            rc = ssd.ssd_backward_varlen(prob, starts, ptr(c["x"]), ptr(c["dt"]), ptr(c["A_log"]), ptr(c["B"]),
                                         ptr(c["C"]), ptr(c["D"]), ptr(c["initial_states"]), ptr(c["dy"]), None,
                                         ptr(c["dx"]), ptr(c["ddt"]), ptr(c["dA_log"]), ptr(c["dB"]), ptr(c["dC"]),
                                         ptr(c["dD"]), None, ptr(ws), wsb, stream.cuda_stream)
        else:
            rc = ssd.ssd_backward(prob, ptr(c["x"]), ptr(c["dt"]), ptr(c["A_log"]), ptr(c["B"]), ptr(c["C"]),
                                  ptr(c["D"]), None, ptr(c["dy"]), None, ptr(c["dx"]), ptr(c["ddt"]),
                                  ptr(c["dA_log"]), ptr(c["dB"]), ptr(c["dC"]), ptr(c["dD"]), None, ptr(ws), wsb,
                                  stream.cuda_stream, events[0].cuda_event if events else None,
                                  events[1].cuda_event if events else None)
        if rc != 0:
            raise ssd.SsdError(rc, "ssd_backward")

    for i in range(args.warmup):
        call(i)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(args.steps):
        call(i)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    if starts is None:
        for i in range(args.steps):
            call(i, kev[i])
        torch.cuda.synchronize()
        ks = sorted(a.elapsed_time(z) for a, z in kev)
        kms = {"mean": sum(ks) / len(ks), "p10": ks[len(ks) // 10], "p50": ks[len(ks) // 2],
               "p90": ks[(9 * len(ks)) // 10]}
    else:   # ssd_backward_varlen takes no events: the whole call's time
        kms = {"mean": ms, "p10": ms, "p50": ms, "p90": ms}
    flops, kbytes, state_bytes, Qb = backward_counts(p)
    compulsory = kbytes
    ksec = kms["mean"] * 1e-3
    tokens = p.batch * p.seqlen
    fast = backward_fast(p)
    if fast:
        t_hbm, t_mfma = kbytes / PEAK_HBM_BPS, flops / PEAK_BF16_FLOPS
        if t_hbm >= t_mfma:
            roof = {"bound": "hbm", "achieved": kbytes / ksec / 1e9, "peak": PEAK_HBM_BPS / 1e9, "unit": "GB/s"}
        else:
            roof = {"bound": "mfma", "achieved": flops / ksec / 1e12, "peak": PEAK_BF16_FLOPS / 1e12,
                    "unit": "TFLOP/s"}
        kname = "k_bwd2_chunk<%d>" % p.dstate if starts is None else "whole call (packed row)"
    else:
        roof = {"bound": "alu", "achieved": flops / ksec / 1e12, "peak": PEAK_F32_VECTOR_FLOPS / 1e12,
                "unit": "TFLOP/s"}
        kname = "k_bwd_chunk"
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = measured_traffic(args.workload, "ssd_backward", BWD_SOURCES)
    roof["kernel"] = kname
    roof["kernel_ms"] = kms
    roof["algorithmic_bytes"] = kbytes
    roof["algorithmic_flops"] = flops
    roof["chunk_state_bytes"] = state_bytes   # design intermediates: in traffic, not in achieved
    print(json.dumps({
        "metric": "SSD bwd tokens/s (gradients of the %s, 1 GPU)" % (
            "2.7B-layer shape" if args.workload == "mamba2_2p7b" else args.workload + " workload"),
        "value": tokens / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16" if fast else p.dtype,
        "data": "synthetic (seeded; Mamba-2 layer shapes)",
        "config": {"workload": "backward_" + args.workload, "batch": p.batch, "seqlen": p.seqlen,
                   "nheads": p.nheads, "headdim": p.headdim, "dstate": p.dstate, "ngroups": p.ngroups,
                   "backward_chunk": Qb},
        "compulsory_bytes": compulsory,
        "hbm_gbps_compulsory": compulsory / (ms * 1e-3) / 1e9,
        "pct_mfma_peak_whole_backward": 100.0 * flops / (ms * 1e-3) / PEAK_BF16_FLOPS if fast else None,
        "roofline": roof,
    }), flush=True)


def block_backward_bench(args, torch, ssd):
    """Gradients of the block at the 2.7B layer shape (ssd_backward_block):
    dt softplus with bias, the layer, the SiLU gate and one-head RMS
    normalisation groups with weight; dout seeded, no initial state, no
    final-state gradient."""
    from paper_2405_21060_amd.inputs import WORKLOADS, make_block_inputs, make_grad_inputs
    from paper_2405_21060_amd.device import act_to_device

    p = WORKLOADS[args.workload]
    bi = make_block_inputs(p, args.seed)
    dout, _ = make_grad_inputs(p, args.seed)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    f32 = lambda a: torch.from_numpy(a).to(dev)
    base = bi.base
    sets = []
    for _ in range(max(1, args.copies)):
        c = {"x": act_to_device(base.x), "dt": act_to_device(bi.dt_raw), "B": act_to_device(base.B),
             "C": act_to_device(base.C), "z": act_to_device(bi.z), "dout": act_to_device(dout)}
        for k in ("x", "dt", "B", "C", "z"):
            c["d" + k] = torch.empty_like(c[k])
        sets.append(c)
    A_log, D, bias, w = f32(base.A_log), f32(base.D), f32(bi.dt_bias), f32(bi.norm_weight)
    dA, dD, dbias, dw = torch.empty_like(A_log), torch.empty_like(D), torch.empty_like(bias), torch.empty_like(w)
    prob = ssd.make_problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size,
                            ssd.SSD_DTYPE_BF16 if p.dtype == "bf16" else ssd.SSD_DTYPE_F32, 0)
    group = p.headdim
    stream = torch.cuda.current_stream(dev)
    ptr = lambda t: None if t is None else t.data_ptr()

    def call(i):
        c = sets[i % len(sets)]
        opts = ssd.make_block_opts(bias, True, 0.0, float("inf"), c["z"], w, group, 1e-5)
        rc = ssd.ssd_backward_block(prob, opts, ptr(c["x"]), ptr(c["dt"]), ptr(A_log), ptr(c["B"]), ptr(c["C"]),
                                    ptr(D), None, ptr(c["dout"]), None, ptr(c["dx"]), ptr(c["ddt"]), ptr(dA),
                                    ptr(c["dB"]), ptr(c["dC"]), ptr(dD), None, ptr(dbias), ptr(c["dz"]), ptr(dw),
                                    ptr(ws), wsb, stream.cuda_stream)
        if rc != 0:
            raise ssd.SsdError(rc, "ssd_backward_block")

    opts0 = ssd.make_block_opts(bias, True, 0.0, float("inf"), sets[0]["z"], w, group, 1e-5)
    wsb = ssd.ssd_backward_block_workspace_bytes(prob, opts0)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    for i in range(args.warmup):
        call(i)
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for i in range(args.steps):
        call(i)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    _, compulsory, _, Qb = backward_counts(p)
    tokens = p.batch * p.seqlen
    act = 2 if p.dtype == "bf16" else 4
    byts = compulsory + 2 * act * tokens * p.nheads * p.headdim + 8 * p.nheads * p.headdim   # z, dz, w, dw
    sec = ms * 1e-3
    print(json.dumps({
        "metric": "SSD block bwd tokens/s (dt softplus + layer + SiLU gate + RMSNorm gradients, 2.7B-layer shape, "
                  "1 GPU)",
        "value": tokens / sec, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": p.dtype, "data": "synthetic (seeded; Mamba-2 layer shapes)",
        "config": {"workload": "block_backward_" + args.workload, "batch": p.batch, "seqlen": p.seqlen,
                   "nheads": p.nheads, "headdim": p.headdim, "dstate": p.dstate, "ngroups": p.ngroups,
                   "norm_group_size": group, "backward_chunk": Qb},
        "roofline": {"bound": "hbm", "achieved": byts / sec / 1e9, "peak": PEAK_HBM_BPS / 1e9, "unit": "GB/s",
                     "frac": byts / sec / PEAK_HBM_BPS, "traffic": None,
                     "kernel": "whole call (forward recomputation, gate/norm and dt steps, layer backward)",
                     "algorithmic_bytes": byts},
    }), flush=True)


def cp_bench(args, torch, ssd):
    """One rank's share of an 8-way sequence split of the 2.7B layer (512 of
    4096 tokens per batch row): the layer from a zero state on the span, the
    span decay and the correction by the state entering the span (the
    exchange of (decay, state) pairs between GPUs is not implemented here;
    the combine of all 8 pairs runs here on one GPU and is timed apart)."""
    from paper_2405_21060_amd.inputs import Problem, make_inputs
    from paper_2405_21060_amd.device import to_device

    R = 8
    p = Problem(4, 4096 // R, 80, 64, 128, 1, 256, "bf16", init_states=True)
    inp = make_inputs(p, args.seed)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sets = [to_device(inp) for _ in range(max(1, args.copies))]
    prob = ssd.make_problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups, p.chunk_size,
                            ssd.SSD_DTYPE_BF16, 0)
    wsb = ssd.ssd_workspace_bytes(prob)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    y = [torch.empty_like(c["x"]) for c in sets]
    fin = torch.empty((p.batch, p.nheads, p.headdim, p.dstate), dtype=torch.float32, device=dev)
    decay = torch.empty((p.batch, p.nheads), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)
    ptr = lambda t: None if t is None else t.data_ptr()
    decays = torch.rand((R, p.batch, p.nheads), device=dev)
    locals_ = torch.randn((R, p.batch, p.nheads, p.headdim, p.dstate), device=dev)

    lib = ssd.load_library()
    import ctypes

    cwsb = ctypes.c_size_t(0)
    lib.ssd_span_correct_workspace_bytes(ctypes.byref(prob), ctypes.byref(cwsb))
    cws = torch.empty(max(int(cwsb.value), 1), dtype=torch.uint8, device=dev)

    def rank_step(i):
        # raw ABI calls (no per-call Python work beyond the calls themselves)
        c = sets[i % len(sets)]
        s_ = stream.cuda_stream
        rc = ssd.ssd_forward(prob, ptr(c["x"]), ptr(c["dt"]), ptr(c["A_log"]), ptr(c["B"]), ptr(c["C"]),
                             ptr(c["D"]), None, None, ptr(y[i % len(sets)]), ptr(fin), ptr(ws), wsb, s_)
        rc = rc or lib.ssd_span_decay(ctypes.byref(prob), ptr(c["dt"]), ptr(c["A_log"]), ptr(decay), s_)
        rc = rc or lib.ssd_span_correct(ctypes.byref(prob), ptr(c["dt"]), ptr(c["A_log"]), ptr(c["C"]),
                                        ptr(c["initial_states"]), ptr(y[i % len(sets)]), ptr(cws),
                                        int(cwsb.value), s_)
        if rc != 0:
            raise ssd.SsdError(rc, "context-parallel rank step")

    def timed(fn):
        for i in range(args.warmup):
            fn(i)
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for i in range(args.steps):
            fn(i)
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / args.steps

    ms = timed(rank_step)
    ms_combine = timed(lambda i: ssd.span_combine(decays, locals_, None))
    tokens = p.batch * p.seqlen
    print(json.dumps({
        "metric": "SSD context-parallel rank share tokens/s (2.7B layer, 8-way sequence split, 1 GPU's span)",
        "value": tokens / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded; Mamba-2 layer shapes)",
        "config": {"workload": "cp8_rank_2p7b", "batch": p.batch, "span": p.seqlen, "ranks": R,
                   "nheads": p.nheads, "headdim": p.headdim, "dstate": p.dstate},
        "combine_8_spans_ms": ms_combine,
        "note": "per rank: layer from a zero state, span decay, entering-state correction",
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=100,
                    help="untimed steps first (the GPU takes on the order of 100 calls to reach its steady clocks)")
    ap.add_argument("--workload", default="mamba2_2p7b")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copies", type=int, default=3)
    ap.add_argument("--kernel-event-every", type=int, default=5,
                    help="forward: time the dominant kernel (events around it) in every n-th timed call")
    ap.add_argument("--no-kernel-events", action="store_true",
                    help="time whole calls only (no events around the dominant kernel)")
    ap.add_argument("--host-offsets", action="store_true",
                    help="packed workloads: time ssd_forward_varlen (host sequence offsets) instead of seq_idx")
    ap.add_argument("--decode", action="store_true",
                    help="time the decode step instead (one token per sequence, batch --decode-batch)")
    ap.add_argument("--decode-batch", type=int, default=256)
    ap.add_argument("--block", action="store_true",
                    help="time the layer with the block steps around it (ssd_forward_block) instead")
    ap.add_argument("--block-norm-group", type=int, default=64)
    ap.add_argument("--backward", action="store_true",
                    help="time the layer's gradients (ssd_backward) instead")
    ap.add_argument("--block-backward", action="store_true",
                    help="time the block's gradients (ssd_backward_block) instead")
    ap.add_argument("--cp-share", action="store_true",
                    help="time one rank's share of an 8-way sequence split instead")
    ap.add_argument("--general-path", action="store_true",
                    help="time the general (per-step) kernels at the workload's shape instead of the fused ones "
                         "(the force_general_path setting of ssd_set_tuning)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="time a plain 1 GiB device-to-device copy instead (reference for the "
                         "FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--gemm-ceiling", action="store_true",
                    help="time a large bf16 matrix product (torch.matmul, 8192^3) instead: the "
                         "box's attainable bf16 matrix-core rate beside the datasheet peak")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py: runs on one GPU only (--gpus 1); the sequence/head "
              "sharding across GPUs is designed but not built", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        n = 1 << 30
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(args.warmup):
            dst.copy_(src)
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(args.steps):
            dst.copy_(src)
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / args.steps
        print(json.dumps({"copy_bytes_each_way": n, "ms": ms, "gbps_read_plus_write": 2 * n / ms / 1e6}),
              flush=True)
        return

    if args.gemm_ceiling:
        n = 8192
        g = torch.Generator(device="cuda:0").manual_seed(args.seed)
        a = torch.randn(n, n, device="cuda:0", generator=g).to(torch.bfloat16)
        b = torch.randn(n, n, device="cuda:0", generator=g).to(torch.bfloat16)
        c = torch.empty(n, n, dtype=torch.bfloat16, device="cuda:0")
        for _ in range(args.warmup):
            torch.matmul(a, b, out=c)
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(args.steps):
            torch.matmul(a, b, out=c)
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / args.steps
        tf = 2.0 * n ** 3 / (ms * 1e-3) / 1e12
        print(json.dumps({"gemm": "bf16 %dx%dx%d torch.matmul" % (n, n, n), "ms": ms, "tflops": tf,
                          "pct_of_bf16_peak": 100.0 * tf * 1e12 / PEAK_BF16_FLOPS}), flush=True)
        return

    from paper_2405_21060_amd import ssd
    from paper_2405_21060_amd.inputs import WORKLOADS, make_inputs
    from paper_2405_21060_amd.device import to_device

    if args.general_path:   # before any workspace is sized: the general kernels need the larger layout
        rc = ssd.ssd_set_tuning("force_general_path", 1)
        if rc != ssd.SSD_OK:
            raise ssd.SsdError(rc, "ssd_set_tuning")

    if args.decode:
        return decode_bench(args, torch, ssd)
    if args.block:
        return block_bench(args, torch, ssd)
    if args.cp_share:
        return cp_bench(args, torch, ssd)
    if args.backward:
        return backward_bench(args, torch, ssd)
    if args.block_backward:
        return block_backward_bench(args, torch, ssd)

    p = WORKLOADS[args.workload]
    inp = make_inputs(p, args.seed)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    copies = [to_device(inp) for _ in range(max(1, args.copies))]
    outs = [torch.empty_like(c["x"]) for c in copies]
    units = inp.nseq if p.varlen else p.batch
    fins = [torch.empty((units, p.nheads, p.headdim, p.dstate), dtype=torch.float32, device=dev)
            for _ in copies]
    prob = ssd.make_problem(p.batch, p.seqlen, p.nheads, p.headdim, p.dstate, p.ngroups,
                            p.chunk_size, ssd.SSD_DTYPE_BF16 if p.dtype == "bf16" else ssd.SSD_DTYPE_F32,
                            inp.nseq if p.varlen else 0)
    wsb = ssd.ssd_workspace_bytes(prob)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)

    # events bracketing the dominant (chunk) kernel of every timed step
    kev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for a, z in kev:  # create the HIP events before their handles are passed down
        a.record(stream)
        z.record(stream)

    starts = None
    if p.varlen and args.host_offsets:
        # packed row with the sequences' host offsets: one forward per sequence
        seq = inp.seq_idx.reshape(-1)
        starts = [0] + [int(v) for v in (seq[1:] != seq[:-1]).nonzero()[0] + 1] + [int(seq.size)]
        wsb = ssd.ssd_forward_varlen_workspace_bytes(prob, starts)
        ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
        args.no_kernel_events = True

    def step(i, events=None):
        c = copies[i % len(copies)]
        ptr = lambda t: None if t is None else t.data_ptr()
        if starts is not None:
            rc = ssd.ssd_forward_varlen(prob, starts, ptr(c["x"]), ptr(c["dt"]), ptr(c["A_log"]), ptr(c["B"]),
                                        ptr(c["C"]), ptr(c["D"]), ptr(c["initial_states"]),
                                        ptr(outs[i % len(copies)]), ptr(fins[i % len(copies)]), ws.data_ptr(),
                                        wsb, stream.cuda_stream)
            if rc != 0:
                raise ssd.SsdError(rc, "ssd_forward_varlen")
            return
        args_ = (prob, ptr(c["x"]), ptr(c["dt"]), ptr(c["A_log"]), ptr(c["B"]), ptr(c["C"]),
                 ptr(c["D"]), ptr(c["initial_states"]), ptr(c["seq_idx"]),
                 ptr(outs[i % len(copies)]), ptr(fins[i % len(copies)]), ws.data_ptr(), wsb,
                 stream.cuda_stream)
        if events is None:
            rc = ssd.ssd_forward(*args_)
        else:
            rc = ssd.ssd_forward_timed(*args_, events[0].cuda_event, events[1].cuda_event)
        if rc != 0:
            raise ssd.SsdError(rc, "ssd_forward")

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    # The timed region: K calls between two events on the launch stream (the
    # whole-job time); inside every n-th call (--kernel-event-every) the
    # library records two more events on that stream right around the dominant
    # (chunk) kernel, which time that kernel alone, live, in the same region.
    # Each such pair costs the call a few microseconds (about 2.5 % of the
    # 2.7B-layer forward when every call carries one), hence the sampling.
    every = max(1, args.kernel_event_every)
    timed_k = [i for i in range(args.steps) if i % every == every - 1] or [args.steps - 1]
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for i in range(args.steps):
        step(i, kev[i] if (not args.no_kernel_events and i in timed_k) else None)
    stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    kms = None
    if not args.no_kernel_events:
        ks = sorted(kev[i][0].elapsed_time(kev[i][1]) for i in timed_k)
        kms = {"mean": sum(ks) / len(ks), "p10": ks[len(ks) // 10], "p50": ks[len(ks) // 2],
               "p90": ks[(9 * len(ks)) // 10], "calls": len(ks)}

    f_full, f_causal, byts = algorithmic_counts(p, inp.nseq)
    sec = ms * 1e-3
    tokens = p.batch * p.seqlen
    peak_flops = PEAK_BF16_FLOPS if p.dtype == "bf16" else PEAK_F32_MFMA_FLOPS
    t_hbm, t_mfma = byts / PEAK_HBM_BPS, f_full / peak_flops
    # Roofline of the dominant kernel: it consumes every compulsory input and
    # produces every output, so its algorithmic bytes per launch are the
    # forward's compulsory bytes (and its FLOPs all but the Gram products).
    ksec = (kms["mean"] if kms else ms) * 1e-3
    if t_hbm >= t_mfma:
        roof = {"bound": "hbm", "achieved": byts / ksec / 1e9, "peak": PEAK_HBM_BPS / 1e9,
                "unit": "GB/s"}
    else:
        roof = {"bound": "mfma", "achieved": f_full / ksec / 1e12, "peak": peak_flops / 1e12,
                "unit": "TFLOP/s"}
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = None if args.general_path else measured_traffic(args.workload)
    roof["kernel"] = dominant_kernel_name(p, args.general_path) + (
        " (whole forward: no kernel events)" if kms is None else "")
    roof["kernel_ms"] = kms
    roof["algorithmic_bytes"] = byts
    line = {
        "metric": "SSD fwd tokens/s (%s, 1 GPU)" % (
            "2.7B-layer shape" if args.workload == "mamba2_2p7b" else args.workload + " workload"),
        "value": tokens / sec,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": p.dtype,
        "data": "synthetic (seeded; shapes and distributions of the Mamba-2 layer)",
        "config": {"workload": args.workload, "batch": p.batch, "seqlen": p.seqlen,
                   "nheads": p.nheads, "headdim": p.headdim, "dstate": p.dstate,
                   "ngroups": p.ngroups, "chunk_size": p.chunk_size,
                   "nseq": inp.nseq if p.varlen else None,
                   "path": "general" if args.general_path else "fused"},
        "tflops_full_block": f_full / sec / 1e12,
        "tflops_causal": f_causal / sec / 1e12,
        "pct_mfma_peak_full_block": 100.0 * f_full / sec / peak_flops,
        "pct_mfma_peak_causal": 100.0 * f_causal / sec / peak_flops,
        "hbm_gbps_compulsory": byts / sec / 1e9,
        "roofline": roof,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(inp)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
