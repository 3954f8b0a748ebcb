"""Benchmark of the GDN chunk forward on one MI355X.

A step is one full pass of the hot path (gates, WY transform, state scan,
output) over one 1280x704 latent frame: B=1, T=3520 tokens (44x80), H=16
heads, Dk=Dv=128, chunk 64, bf16 q/k/v with an fp32 state carried in and out.
The inputs are seeded synthetic tensors already resident in HBM; the workspace
is preallocated, so the timed region only enqueues the path's kernels (on this
workload two: the WY kernel and the state scan with the output fused into it).

Prints ONE JSON line.  Besides throughput it reports the roofline of the
dominant kernel (per-stage durations from HIP events recorded on the stream
the kernels run on) and, on rank 0, the fp64 CPU oracle timed on the host
cores as a reported baseline.

``--path frame`` measures the frame-wise forward instead (one decay per frame,
all tokens of a frame written at once): a step is one streaming call of 3
latent frames of 44x80 tokens, B=1, F=3, N=3520, H=16, Dk=Dv=128, bf16, with
the fp32 state carried in and out; its four kernels are the frame summaries,
their reduction over token splits, the scan over frames and the output.
``--path frame-norm`` measures the same call with the normalizer state and the
normalized readout (non-negative feature maps); ``--path frame-bidir`` and
``--path frame-bidir-norm`` the bidirectional form of either (a backward scan
over the call's frames beside the forward one); ``--path frame-fused`` (and
``frame-fused-bidir``) the whole operator of the paper's GDN block around it:
raw q and k projections through RMSNorm, ReLU and 3D RoPE, the two states,
the normalized readout, the SiLU gate and the per-head projection W_o.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import gdn_inputs  # noqa: E402

METRIC = "GDN fwd tokens/sec and TFLOP/s at T=3520,H=16,D=128 bf16; % of MFMA peak"
WORKLOAD = 1                 # one 1280x704 frame
PEAK_BF16_TFLOPS = 2516.6    # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3      # MI355X fp32 matrix
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E
# stage name (as the library reports stages) -> kernel
KERNELS = {"wy": "gdn_wy_kernel", "group_transfer": "gdn_chunkscan_kernel<SCAN_TRANS>",
           "group_scan": "gdn_groupscan_kernel", "chunk_states": "gdn_chunkscan_kernel<SCAN_STATES>",
           "output": "gdn_output_kernel"}
KERNELS_FUSED = dict(KERNELS, chunk_states="gdn_chunkscan_kernel<SCAN_STATES, output fused>")
EXTRA_WORKLOADS = (0, 2, 3, 4)
# committed counter summaries of the token path, per workload
TRAFFIC_SUMMARY = {1: "traffic_frame1280x704.json", 2: "traffic_stream3x1280x704.json",
                   4: "traffic_long12x1280x704.json"}


def path_counts(B, T, H, Dk, Dv, C=64, esz=2):
    """The path's algorithmic work and I/O (the chunked method's own contractions,
    causal and strict triangles counted once; every input read once, every output
    written once, the state in and out):
        F_alg = 6 Dk Dv + (C-1)(2Dk+Dv) + (C+1)(Dk+Dv) + C^2/3   flop per token-head
        bytes = (2Dk+Dv) s + 8 + Dv s                            per token-head
                + 2 B H Dk Dv 4                                  per call (fp32 state)
    with s the q/k/v/out element size.  Workspace traffic is not algorithmic."""
    n = B * T * H
    flops = n * (6.0 * Dk * Dv + (C - 1) * (2 * Dk + Dv) + (C + 1) * (Dk + Dv) + C * C / 3.0)
    io = n * ((2 * Dk + Dv) * esz + 8 + Dv * esz) + 2 * B * H * Dk * Dv * 4
    return flops, io


def workspace_traffic(B, T, H, Dk, Dv, G, C=64, esz=2):
    """Workspace bytes each stage writes and reads (every byte once).  The WY
    kernel writes the gates (g, and a record of the per-token key decay factors
    in fp32 with g_C), -W and U~t; the scans read the keys from the input.  With one scan
    group on the bf16 path the output is fused into the scan: the WY kernel then
    also writes the decay-scaled queries and the masked decayed Q K^T tile of
    every chunk (row fragments the scan's output waves read) and the scan
    writes no per-chunk state."""
    NC = -(-T // C)
    NG = -(-NC // G)
    nch = B * H * NC
    fused = esz == 2 and NG == 1
    ngr = B * H * NG if NG > 1 else 0
    gates = nch * (C * 8 + (C + 4) * 4)
    fac = nch * C * (Dk + Dv) * esz                        # -W, U~t
    scan_gates = nch * (C + 4) * 4                         # key scales, g_C
    qp = nch * C * (Dk + C) * esz if fused else 0          # scaled Q, masked P
    grp = ngr * (Dk * Dk * esz + Dv * Dk * 4 + 8)          # N, Psi^T, log Gamma
    hg = ngr * Dv * Dk * 4                                 # group entry states
    hs_us = 0 if fused else nch * Dv * (Dk + C) * esz      # per-chunk state and pseudo-values
    zero = {"written": 0, "read": 0}
    return {"wy": {"written": gates + fac + qp, "read": 0},
            "group_transfer": {"written": grp, "read": fac + scan_gates} if ngr else zero,
            "group_scan": {"written": hg, "read": grp} if ngr else zero,
            "chunk_states": {"written": hs_us, "read": fac + scan_gates + hg + qp},
            "output": zero if fused else {"written": 0, "read": hs_us + nch * C * 8}}


def pct(xs, p):
    return float(np.percentile(np.asarray(xs, dtype=np.float64), p))


def stats(xs):
    return {"median": round(pct(xs, 50), 5), "p10": round(pct(xs, 10), 5), "p90": round(pct(xs, 90), 5)}


def host_threads():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(inp, B, T, min_seconds=10.0):
    """Time the fp64 oracle (as it stands) on whole workload calls for ~10 s."""
    import oracle
    threads = host_threads()
    reps, elapsed = 0, 0.0
    while elapsed < min_seconds and reps < 1000:
        t0 = time.perf_counter()
        oracle.gdn_forward(inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"],
                           inp["state_in"], nthreads=threads)
        elapsed += time.perf_counter() - t0
        reps += 1
    return {"value": B * T * reps / elapsed, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{reps} whole calls of the timed workload (B={B}, T={T}, H=16, D=128), "
                      f"fp64 token recurrence, {elapsed:.1f} s"}


def load_traffic(summary):
    """Per-stage HBM bytes per launch from a committed counter summary, or None when
    the summary is missing or was taken on different kernel source."""
    path = os.path.join(ROOT, "profiles", summary)
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
        import hashlib
        h = hashlib.sha256()
        for f in rec["sources"]:
            h.update(open(os.path.join(ROOT, f), "rb").read())
        if h.hexdigest() != rec["source_sha256"]:
            return None
        return {k: float(v["hbm_bytes_per_launch"]) for k, v in rec["stages"].items()}
    except Exception:
        return None


def token_roofline(flops, io, names, kernels, traffic, peak_tflops, own_io=None):
    """Roofline of the dominant kernel.  Token path: the call's algorithmic I/O
    (or flops) over that kernel's launch duration.  Frame-wise paths (own_io
    given): the dominant kernel's own share of the call's I/O -- the inputs it
    reads and the outputs it writes, no workspace.  The paths' intensity is
    below the ridge (~315 flop/B), so their bound is HBM."""
    dom = max(names, key=names.get)
    sec = names[dom] / 1e3
    if own_io is not None:
        io = own_io[dom]
    bound_hbm = flops / io < peak_tflops * 1e12 / (PEAK_HBM_GBS * 1e9)
    a_gbs = io / sec / 1e9
    a_tf = flops / sec / 1e12
    r = {"bound": "hbm", "achieved": round(a_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
         "frac": round(a_gbs / PEAK_HBM_GBS, 4)} if bound_hbm else \
        {"bound": "mfma", "achieved": round(a_tf, 2), "peak": peak_tflops, "unit": "TFLOP/s",
         "frac": round(a_tf / peak_tflops, 4)}
    call_traffic = None if traffic is None else sum(traffic.get(k, 0.0) for k in names if names[k] > 0)
    r.update({"traffic": None if call_traffic is None else round(call_traffic),
              "traffic_scope": "whole call (sum over the call's kernels), FETCH_SIZE and WRITE_SIZE "
                               "scaled by a plain copy kernel",
              "traffic_over_algorithmic": None if call_traffic is None else round(call_traffic / io, 3),
              "traffic_dominant_kernel": None if traffic is None or dom not in traffic else round(traffic[dom]),
              "kernel": kernels.get(dom, dom), "duration_ms": round(names[dom], 5),
              "algorithmic_bytes_per_launch": io, "algorithmic_flops_per_launch": flops,
              "mfma_frac_dominant": round(a_tf / peak_tflops, 4)})
    return r


def time_steps(step, stream, steps, warmup, torch):
    """`warmup` untimed steps, then `steps` steps between two events on `stream`
    (bracketed by synchronizations): the mean.  Then the same number of steps
    again, each between its own pair of events: the per-step durations in ms
    (their median and spread; the events between steps add a little time, so
    the mean is taken from the first pass)."""
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    mean = e0.elapsed_time(e1) / steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        a.record(stream)
        step()
        b.record(stream)
    torch.cuda.synchronize()
    return mean, [a.elapsed_time(b) for a, b in ev]


def run_extra_workload(idx, gdn, torch, dev, stream, reps):
    """GPU time per call on workload `idx` (device-drawn inputs of its shapes and
    value distributions; workload 2 is the 20-call streaming chain with the state
    threaded on the device, timed as a whole and divided by 20)."""
    w = gdn_inputs.WORKLOADS[idx]
    esz = 2 if w.dtype == "bf16" else 4
    calls = [gdn_inputs.make_device_inputs(idx, dev, call=c) for c in range(w.calls)]
    B, T, H, Dk, Dv = w.B, w.T, w.H, w.Dk, w.Dv
    out = torch.empty((B, T, H, Dv), dtype=calls[0]["q"].dtype, device=dev)
    st = [torch.zeros((B, H, Dk, Dv), dtype=torch.float32, device=dev) for _ in range(2)]
    if calls[0]["state_in"] is not None:
        st[0].copy_(calls[0]["state_in"])
    ws = gdn.workspace(calls[0]["q"], calls[0]["v"])
    fwd = gdn.gdn_chunk_forward_ws if w.dtype == "bf16" else gdn.gdn_chunk_forward_f32_ws

    def chain():
        for c, inp in enumerate(calls):
            si = st[c & 1] if (c > 0 or calls[0]["state_in"] is not None) else None
            fwd(inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], si, out, st[(c + 1) & 1], ws,
                stream=stream)

    _, per = time_steps(chain, stream, reps, 2, torch)
    per_call = [x / w.calls for x in per]
    inp = calls[0]
    stage = gdn.gdn_profile_stages(inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], inp["state_in"],
                                   out, st[1], ws, reps=max(3, reps // 2), stream=stream)
    torch.cuda.synchronize()
    names = {k: v for k, v in zip(gdn.STAGE_NAMES, stage) if v > 0}
    G = gdn.gdn_scan_group_size(B, H, T, Dk, Dv, is_bf16=esz == 2)
    fused = esz == 2 and -(-(-(-T // 64)) // G) == 1
    flops, io = path_counts(B, T, H, Dk, Dv, esz=esz)
    wst = workspace_traffic(B, T, H, Dk, Dv, G, esz=esz)
    ws_bytes = sum(v["written"] + v["read"] for v in wst.values())
    med = pct(per_call, 50) / 1e3
    peak = PEAK_BF16_TFLOPS if esz == 2 else PEAK_F32_TFLOPS
    dom = max(names, key=names.get)
    rec = {"workload": w.name, "calls": w.calls, "ms_per_call": stats(per_call),
           "tokens_per_s": round(B * T / med, 1), "tflops": round(flops / med / 1e12, 3),
           "mfma_frac": round(flops / med / 1e12 / peak, 5), "peak_tflops": peak,
           "hbm_frac_io": round(io / med / 1e9 / PEAK_HBM_GBS, 4),
           "algorithmic_bytes": io, "algorithmic_flops": flops,
           "scan_group": G, "output_fused": fused,
           "stage_ms": {k: round(v, 5) for k, v in names.items()},
           "dominant_kernel": (KERNELS_FUSED if fused else KERNELS).get(dom, dom),
           "workspace_bytes": ws_bytes,
           "workspace_gbs": round(ws_bytes / med / 1e9, 1)}
    del calls, out, st, ws
    torch.cuda.empty_cache()
    return rec


FRAME_METRIC = ("frame-wise GDN fwd tokens/sec and TFLOP/s at F=3 frames x N=3520 tokens, "
                "H=16, D=128 bf16")
FRAME_NORM_METRIC = ("frame-wise normalized GDN fwd tokens/sec and TFLOP/s at F=3 frames x N=3520 tokens, "
                     "H=16, D=128 bf16")
FRAME_BIDIR_METRIC = ("bidirectional frame-wise GDN fwd tokens/sec and TFLOP/s at F=3 frames x N=3520 tokens, "
                      "H=16, D=128 bf16")
FRAME_BIDIR_NORM_METRIC = ("bidirectional frame-wise normalized GDN fwd tokens/sec and TFLOP/s at F=3 frames x "
                           "N=3520 tokens, H=16, D=128 bf16")
FRAME_FUSED_METRIC = ("fused frame-wise GDN operator (RMSNorm/ReLU/3D-RoPE prologue, SiLU gate and W_o epilogue) "
                      "fwd tokens/sec and TFLOP/s at F=3 frames x N=3520 tokens, H=16, D=128 bf16")
FRAME_KERNELS = {"summaries": "gdn_frame_summary_kernel", "reduce": "gdn_frame_reduce_kernel",
                 "scan": "gdn_frame_scan_kernel", "output": "gdn_frame_output_kernel"}


def frame_algorithmic_counts(B, F, N, H, Dk, Dv, NS, esz=2, norm=False, bidir=False, fused=False):
    """See below; with fused and esz = 4 (the fp32 operator) the workspace also
    carries the four feature maps (written once, each read once) and the gated
    readout (written and read once)."""
    r = _frame_counts(B, F, N, H, Dk, Dv, NS, esz, norm, bidir, fused)
    if fused and esz == 4:
        n = B * F * N * H
        r["workspace"]["summaries"]["written"] += 4 * n * Dk * 4
        r["workspace"]["summaries"]["read"] += 2 * n * Dk * 4
        r["workspace"]["output"]["read"] += 2 * n * Dk * 4 + n * Dv * 4
        r["workspace"]["output"]["written"] += n * Dv * 4
    return r


def _frame_counts(B, F, N, H, Dk, Dv, NS, esz, norm, bidir, fused):
    """Algorithmic flops per stage and the call's I/O bytes for the frame-wise path,
    plus each stage's workspace bytes (reported apart: not algorithmic).

    flops: summaries G = K^T B K and A = K^T B V over every token (plus b = K^T beta
    for the normalizer, and the unrotated-key Gram matrix of the fused operator);
    scan H_f = alpha (H - G H) + A per frame (z as one more column with the
    normalizer; the backward scan over the F - 1 later frames when bidirectional);
    output O = Q H_f per token (d = Q z with the normalizer; W_o in the fused
    operator).  The token-split reduction adds no algorithmic flops.
    I/O bytes: q, k, v, out (and the fused operator's gate and W_o), alpha, beta,
    the state (and z) in and out."""
    if fused:
        norm = True
    Dz = 1 if norm else 0               # normalizer columns that are work
    Ds = Dv + (16 if norm else 0)       # state columns the kernels carry
    n = B * F * N * H                   # token-heads
    u = B * H * F                       # (frame, head) units
    st = B * H * Dk * Dv * 4 + (B * H * Dk * 4 if norm else 0)
    # a split's Gram partials: the 16 x 16 tiles on and above the diagonal
    R = Dk // 16
    gram = R * (R + 1) // 2 * 256 * 4
    part = u * NS * (gram + Dk * Ds * 4) if NS > 1 else 0
    f = {"summaries": 2.0 * n * Dk * (Dk + Dv + Dz),
         "reduce": 0.0,
         "scan": u * (2.0 * Dk * Dk * (Dv + Dz) + 3.0 * Dk * (Dv + Dz)),
         "output": 2.0 * n * Dk * (Dv + Dz) + (n * Dv if norm else 0)}
    ws = {"summaries": {"written": part if NS > 1 else u * (Dk * Dk * esz + Dk * Ds * 4), "read": 0},
          "reduce": {"written": u * (Dk * Dk * esz + Dk * Ds * 4) if NS > 1 else 0, "read": part},
          "scan": {"written": u * Dk * Ds * esz, "read": u * (Dk * Dk * esz + Dk * Ds * 4)},
          "output": {"written": 0, "read": u * Dk * Ds * esz}}
    if fused:
        gpart = u * NS * gram if NS > 1 else 0
        f["summaries"] += 2.0 * n * Dk * Dk
        ws["summaries"]["written"] += gpart if NS > 1 else u * Dk * Dk * esz
        ws["reduce"]["read"] += gpart
        ws["reduce"]["written"] += u * Dk * Dk * esz if NS > 1 else 0
        ws["scan"]["read"] += u * Dk * Dk * esz
        f["output"] += 2.0 * n * Dv * Dv
    if bidir:
        ub = B * H * (F - 1)
        f["scan"] += ub * (2.0 * Dk * Dk * (Dv + Dz) + 3.0 * Dk * (Dv + Dz)) + u * Dk * (Dv + Dz)
        ws["scan"]["written"] += u * Dk * Ds * 4
        ws["scan"]["read"] += u * Dk * Ds * 4
    io_bytes = n * ((2 * Dk + 2 * Dv) * esz + 4) + u * 4 + 2 * st
    # each kernel's own share of the call's I/O
    own = {"summaries": n * ((Dk + Dv) * esz + 4), "reduce": 0,
           "scan": u * 4 + 2 * st, "output": n * (Dk + Dv) * esz}
    if fused:
        io_bytes += n * Dv * esz + H * Dv * Dv * esz
        own["output"] += n * Dv * esz + H * Dv * Dv * esz
    return dict(flops=f, io_bytes=io_bytes, workspace=ws, own_io=own)


def frame_cpu_baseline(inp, B, T, H, Dk, min_seconds=10.0, norm=False, bidir=False, fused=False):
    """Time the fp64 frame-wise oracle (as it stands) on whole calls for ~10 s."""
    import oracle
    threads = host_threads()
    reps, elapsed = 0, 0.0
    if fused:
        while elapsed < min_seconds and reps < 1000:
            t0 = time.perf_counter()
            oracle.gdn_frame_forward_fused(inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], inp["gate"],
                                           inp["w_o"], inp["state_in"], inp["z_in"],
                                           frame_tokens=inp["frame_tokens"], gain_q=inp["gain_q"],
                                           gain_k=inp["gain_k"], rope_freq=inp["rope_freq"],
                                           rope_axis=inp["rope_axis"], lat_w=inp["lat_w"], t0=inp["t0"],
                                           bidirectional=bidir, nthreads=threads)
            elapsed += time.perf_counter() - t0
            reps += 1
        return {"value": B * T * reps / elapsed, "unit": "tokens/s", "cores": threads, "kind": "oracle",
                "cpu_model": cpu_model(),
                "sample": f"{reps} whole calls of the timed workload (B={B}, T={T}, H={H}, D={Dk}), "
                          f"fp64 fused operator{' (bidirectional)' if bidir else ''}, {elapsed:.1f} s"}
    extra = dict(normalized=True, z_in=inp["z_in"]) if norm else {}
    if bidir:
        extra["bidirectional"] = True
    while elapsed < min_seconds and reps < 1000:
        t0 = time.perf_counter()
        oracle.gdn_frame_forward(inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"],
                                 inp["state_in"], frame_tokens=inp["frame_tokens"], nthreads=threads,
                                 **extra)
        elapsed += time.perf_counter() - t0
        reps += 1
    return {"value": B * T * reps / elapsed, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"{reps} whole calls of the timed workload (B={B}, T={T}, H={H}, D={Dk}), "
                      f"fp64 {'bidirectional ' if bidir else ''}frame-wise recurrence, {elapsed:.1f} s"}


def run_frame(args, torch, gdn, dev, to_dev, timed, norm=False, bidir=False, fused=False, f32=False):
    F, N = 3, 3520
    if fused:
        norm = True
        inp = gdn_inputs.make_fused_inputs(2, F, frame_tokens=N, state="normal0.02", lat_w=80, t0=0,
                                           dtype="f32" if f32 else "bf16")
    else:
        inp = gdn_inputs.make_frame_inputs(2, F, frame_tokens=N, state="normal0.02",
                                           features="relu" if norm else "gauss")
    B, T, H, Dk = inp["q"].shape
    Dv = inp["v"].shape[-1]
    q, k, v = to_dev(inp["q"]), to_dev(inp["k"]), to_dev(inp["v"])
    alpha, beta, s_in = to_dev(inp["alpha"]), to_dev(inp["beta"]), to_dev(inp["state_in"])
    out = torch.empty((B, T, H, Dv), dtype=q.dtype, device=dev)
    s_out = torch.empty((B, H, Dk, Dv), dtype=torch.float32, device=dev)
    z_in = to_dev(inp["z_in"]) if norm else None
    fz = {key: to_dev(inp[key]) for key in ("gate", "w_o", "gain_q", "gain_k", "rope_freq", "rope_axis")} if fused \
        else None
    z_out = torch.empty((B, H, Dk), dtype=torch.float32, device=dev) if norm else None
    ts = args.token_splits
    ws = gdn.fused_workspace(q, v, N, ts) if fused else gdn.frame_workspace(q, v, N, ts)
    NS = gdn.gdn_frame_token_splits(B, H, F, N, Dk, Dv, ts)
    stream = torch.cuda.current_stream(dev)

    def step():
        if fused:
            gdn.frame_forward_fused(q, k, v, fz["gate"], fz["w_o"], alpha, beta, fz["gain_q"], fz["gain_k"],
                                    fz["rope_freq"], fz["rope_axis"], s_in, z_in, frame_tokens=N, lat_w=80, t0=0,
                                    bidirectional=bidir, out=out, state_out=s_out, z_out=z_out, ws=ws,
                                    token_splits=ts, stream=stream)
        elif bidir:
            gdn.frame_forward_bidir(q, k, v, alpha, beta, s_in, z_in, frame_tokens=N, normalized=norm, out=out,
                                    state_out=s_out, z_out=z_out, ws=ws, token_splits=ts, stream=stream)
        elif norm:
            gdn.frame_forward_norm(q, k, v, alpha, beta, s_in, z_in, frame_tokens=N, out=out,
                                   state_out=s_out, z_out=z_out, ws=ws, token_splits=ts, stream=stream)
        else:
            gdn.gdn_frame_forward_ex(q, k, v, alpha, beta, s_in, out, s_out, ws, N, token_splits=ts,
                                     stream=stream)

    ms_per_step, per_step, cold = timed(step, stream)
    if fused:
        stage_ms = gdn.gdn_frame_profile_stages_fused(q, k, v, fz["gate"], fz["w_o"], alpha, beta, fz["gain_q"],
                                                      fz["gain_k"], fz["rope_freq"], fz["rope_axis"], s_in, z_in, out,
                                                      s_out, z_out, ws, N, 80, 0, bidirectional=bidir,
                                                      token_splits=ts, reps=args.steps, stream=stream)
    elif bidir:
        stage_ms = gdn.gdn_frame_profile_stages_bidir(q, k, v, alpha, beta, s_in, z_in, out, s_out, z_out,
                                                      ws, N, normalized=norm, token_splits=ts, reps=args.steps,
                                                      stream=stream)
    elif norm:
        stage_ms = gdn.gdn_frame_profile_stages_norm(q, k, v, alpha, beta, s_in, z_in, out, s_out, z_out,
                                                     ws, N, token_splits=ts, reps=args.steps,
                                                     stream=stream)
    else:
        stage_ms = gdn.gdn_frame_profile_stages(q, k, v, alpha, beta, s_in, out, s_out, ws, N,
                                                token_splits=ts, reps=args.steps, stream=stream)
    names = {k_: v_ for k_, v_ in zip(gdn.FRAME_STAGE_NAMES, stage_ms) if v_ > 0}
    torch.cuda.synchronize()
    esz = 4 if f32 else 2
    cnt = frame_algorithmic_counts(B, F, N, H, Dk, Dv, NS, esz=esz, norm=norm, bidir=bidir, fused=fused)
    flops = sum(cnt["flops"].values())
    sec = ms_per_step / 1e3
    tflops = flops / sec / 1e12
    # counter summaries: the bidirectional form shares every kernel but the scan
    # with the unidirectional one
    summary = ("traffic_frames3x1280x704_fused.json" if fused else
               "traffic_frames3x1280x704_norm.json" if norm else "traffic_frames3x1280x704.json")
    traffic = None if f32 else load_traffic(summary)
    if traffic is not None and bidir:
        traffic = None
    kernels = dict(FRAME_KERNELS)
    if fused and f32:
        kernels.update({"summaries": "gdn_frame_features_kernel + 2 x gdn_frame_summary_kernel<float>",
                        "output": "gdn_frame_output_f32_fused_kernel + gdn_frame_project_f32_kernel"})
    elif fused:
        kernels.update({"summaries": "gdn_frame_summary_fused_kernel", "output": "gdn_frame_output_fused_kernel"})
    peak = PEAK_F32_TFLOPS if f32 else PEAK_BF16_TFLOPS
    roofline = token_roofline(flops, cnt["io_bytes"], names, kernels, traffic, peak, own_io=cnt["own_io"])
    rec = {
        "metric": (FRAME_FUSED_METRIC.replace(" bf16", " fp32") if f32 else FRAME_FUSED_METRIC)
                  + (" (bidirectional)" if bidir else "") if fused
                  else (FRAME_BIDIR_NORM_METRIC if norm else FRAME_BIDIR_METRIC) if bidir
                  else (FRAME_NORM_METRIC if norm else FRAME_METRIC),
        "value": round(B * T / sec, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if f32 else "bf16",
        "data": "synthetic",
        "config": {"workload": "frame-wise streaming call of 3 latent 1280x704 frames: B=1 F=3 "
                               "N=3520 (44x80) H=16 Dk=Dv=128, " + ("fp32" if f32 else "bf16") +
                               " q/k/v, one decay per frame, "
                               "key scale 1/sqrt(Dk N), fp32 state in/out"
                               + ("; normalizer state in/out and normalized readout (eps 1e-6), "
                                  "non-negative (ReLU) feature maps" if norm and not fused else "")
                               + ("; fused operator: raw q/k projections through RMSNorm, ReLU and a fixed 3D "
                                  "RoPE (44x80 latent grid), normalizer from the unrotated keys, SiLU output gate "
                                  "and per-head W_o" if fused else "")
                               + ("; bidirectional (forward scan from the state plus a backward scan over "
                                  "the call's frames from zero)" if bidir else ""),
                   "B": B, "F": F, "N": N, "T": T, "H": H, "Dk": Dk, "Dv": Dv, "token_splits": NS},
        "tflops": round(tflops, 2),
        "mfma_frac": round(tflops / peak, 4),
        "hbm_frac_io": round(cnt["io_bytes"] / sec / 1e9 / PEAK_HBM_GBS, 4),
        "step_ms": stats(per_step),
        "ms_per_step_cold": None if cold is None else stats(cold),
        "stage_ms": {k_: round(v_, 5) for k_, v_ in names.items()},
        "workspace_bytes": cnt["workspace"],
        "roofline": roofline,
    }
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = frame_cpu_baseline(inp, B, T, H, Dk, norm=norm, bidir=bidir, fused=fused)
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing leg")
    ap.add_argument("--workload", type=int, default=WORKLOAD, choices=range(len(gdn_inputs.WORKLOADS)),
                    help="token path: the workload a step runs (default 1, one 1280x704 frame; the "
                         "others draw their inputs on the device)")
    ap.add_argument("--no-workloads", action="store_true",
                    help="token path: skip the per-call timing of the other four workloads")
    ap.add_argument("--cold-steps", type=int, default=20,
                    help="extra steps each preceded by a 1 GiB write that evicts the caches")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB first (a known-size "
                         "reference for hardware traffic counters)")
    ap.add_argument("--path", choices=("token", "frame", "frame-norm", "frame-bidir", "frame-bidir-norm",
                                       "frame-fused", "frame-fused-bidir", "frame-fused-f32",
                                       "frame-fused-f32-bidir"),
                    default="token",
                    help="token: the token-wise chunk forward (default); frame: the frame-wise "
                         "forward; frame-norm: the frame-wise forward with the normalizer; "
                         "frame-bidir(-norm): their bidirectional forms; frame-fused(-bidir): the whole "
                         "operator with its prologue and epilogue; frame-fused-f32(-bidir): its fp32 mode")
    ap.add_argument("--token-splits", type=int, default=0,
                    help="frame path: token splits per frame (0 = the library's choice)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the (b, h) streams shard across GPUs with no communication, so the one-GPU "
              "number is the per-GPU figure).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2605_30409_amd as gdn

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)

    def to_dev(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib << 18  # float32 elements
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    def timed(step, stream):
        """Warmup, then `steps` timed steps (an event before each and after the last,
        on `stream`), then cold-cache steps (each after a 1 GiB write that evicts L2
        and the MALL).  Returns (mean ms per step, per-step ms, cold per-step ms)."""
        ms, per = time_steps(step, stream, args.steps, args.warmup, torch)
        cold = None
        if args.cold_steps > 0:
            scratch = torch.empty(1 << 28, dtype=torch.float32, device=dev)
            cold = []
            for i in range(args.cold_steps):
                scratch.fill_(float(i))
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                step()
                b.record(stream)
                torch.cuda.synchronize()
                cold.append(a.elapsed_time(b))
            del scratch
        return ms, per, cold

    if args.path.startswith("frame"):
        run_frame(args, torch, gdn, dev, to_dev, timed, norm=args.path.endswith("-norm"),
                  bidir="-bidir" in args.path, fused="-fused" in args.path, f32="-f32" in args.path)
        return

    widx = args.workload
    w = gdn_inputs.WORKLOADS[widx]
    B, T, H, Dk, Dv, C = w.B, w.T, w.H, w.Dk, w.Dv, w.chunk
    bf16 = w.dtype == "bf16"
    if widx == WORKLOAD:
        inp = gdn_inputs.make_inputs(WORKLOAD)
        calls = [{key: to_dev(inp[key]) for key in ("q", "k", "v", "alpha", "beta", "state_in")}]
    else:
        # device-drawn inputs (timing only); the streaming workload's calls
        # each get their own draw and the state is threaded through them
        inp = None
        calls = [gdn_inputs.make_device_inputs(widx, dev, call=c) for c in range(w.calls)]
    out = torch.empty((B, T, H, Dv), dtype=calls[0]["q"].dtype, device=dev)
    s_out = torch.empty((B, H, Dk, Dv), dtype=torch.float32, device=dev)
    states = [torch.zeros_like(s_out), s_out]
    ws = gdn.workspace(calls[0]["q"], calls[0]["v"])
    stream = torch.cuda.current_stream(dev)
    fwd = gdn.gdn_chunk_forward_ws if bf16 else gdn.gdn_chunk_forward_f32_ws
    ncall = [0]

    def step():
        c = ncall[0]
        x = calls[c % len(calls)]
        if len(calls) == 1:
            fwd(x["q"], x["k"], x["v"], x["alpha"], x["beta"], x["state_in"], out, s_out, ws, chunk=C, stream=stream)
        else:
            fwd(x["q"], x["k"], x["v"], x["alpha"], x["beta"], states[c & 1], out, states[(c + 1) & 1], ws, chunk=C,
                stream=stream)
        ncall[0] = c + 1

    ms_per_step, per_step, cold = timed(step, stream)
    x = calls[0]
    q, k, v, alpha, beta = x["q"], x["k"], x["v"], x["alpha"], x["beta"]
    s_in = x["state_in"] if x["state_in"] is not None else states[0]

    # Per-stage durations: HIP events recorded by the library on the same stream.
    stage_ms = gdn.gdn_profile_stages(q, k, v, alpha, beta, s_in, out, s_out, ws,
                                      reps=args.steps, chunk=C, stream=stream)
    names = {k_: v_ for k_, v_ in zip(gdn.STAGE_NAMES, stage_ms) if v_ > 0}
    torch.cuda.synchronize()

    G = gdn.gdn_scan_group_size(B, H, T, Dk, Dv, C, is_bf16=bf16)
    NG = -(-(-(-T // C)) // G)
    fused = bf16 and NG == 1
    esz = 2 if bf16 else 4
    flops, io = path_counts(B, T, H, Dk, Dv, C, esz=esz)
    sec = ms_per_step / 1e3
    tflops = flops / sec / 1e12
    peak = PEAK_BF16_TFLOPS if bf16 else PEAK_F32_TFLOPS
    traffic = load_traffic(TRAFFIC_SUMMARY.get(widx, "none"))
    roofline = token_roofline(flops, io, names, KERNELS_FUSED if fused else KERNELS, traffic, peak)

    rec = {
        "metric": METRIC if widx == WORKLOAD else f"GDN fwd tokens/sec and TFLOP/s, workload {w.name}",
        "value": round(B * T / sec, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": "one 1280x704 latent frame: B=1 T=3520 (44x80) H=16 Dk=Dv=128 "
                               "chunk=64, bf16 q/k/v, fp32 state in/out" if widx == WORKLOAD else w.name
                               + (f" (a step is one call of the {w.calls}-call chain, state threaded)"
                                  if w.calls > 1 else ""),
                   "B": B, "T": T, "H": H, "Dk": Dk, "Dv": Dv, "chunk": C,
                   "scan_group": G, "scan_groups": NG, "output_fused": fused},
        "step_ms": stats(per_step),
        "tflops": round(tflops, 2),
        "mfma_frac": round(tflops / peak, 4),
        "hbm_frac_io": round(io / sec / 1e9 / PEAK_HBM_GBS, 4),
        "ms_per_step_cold": None if cold is None else stats(cold),
        "stage_ms": {k_: round(v_, 5) for k_, v_ in names.items()},
        "workspace_bytes": workspace_traffic(B, T, H, Dk, Dv, G, C, esz=esz),
        "roofline": roofline,
    }
    if not args.no_workloads and widx == WORKLOAD:
        extra = {}
        for idx in EXTRA_WORKLOADS:
            extra[str(idx)] = run_extra_workload(idx, gdn, torch, dev, stream, reps=10 if idx == 4 else 20)
        rec["workloads"] = extra
    if not args.no_cpu_baseline and inp is not None:
        rec["cpu_baseline"] = cpu_baseline(inp, B, T)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
