"""Seeded synthetic inputs for the GDN chunk forward.

This module is shared by the tests, the benchmark and the smoke check.  It
holds no part of the method's arithmetic: it only draws random tensors of the
shapes and value distributions of the five workloads below, and rounds them to
the storage type.  Both the HIP path and the fp64 oracle read the very same
stored arrays.

Recipe (PCG64 via ``numpy.random.default_rng(seed)``, seed = 1000 * workload
+ call index, draws in this order):
  q, k ~ N(0, 1) in fp32, each (b, t, h) row L2-normalised over D in fp32,
  v ~ N(0, 1), the alpha noise, the beta noise, then state_in; bf16 workloads
  round q, k, v to bf16 with round-to-nearest-even after normalising.

The tokens stand in for DiT activations of 1280x704 video: a latent frame is a
44 x 80 token grid (3520 tokens), a streaming chunk is 3 frames.  The decay
alpha follows the Mamba-2 style exp(-softplus(.)) shape of the paper's decay
gate (equation appendix_gdn_alpha) and beta the sigmoid of its write gate
(equation appendix_gdn_beta); the weights producing them are not part of this
path, so their pre-activations are drawn as Gaussians.
"""
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    T: int
    H: int
    Dk: int
    Dv: int
    dtype: str          # "f32" or "bf16" for q, k, v and out
    alpha: str          # "softplus0", "softplus2" or "uniform0.5"
    beta: str           # "sigmoid" or "uniform"
    state: str          # "zero" or "normal0.02"
    calls: int = 1
    chunk: int = 64


WORKLOADS = (
    Workload("tiny-f32 B1 T256 H2 D64", 1, 256, 2, 64, 64, "f32",
             "softplus0", "sigmoid", "zero"),
    Workload("frame-1280x704 B1 T3520 H16 D128", 1, 3520, 16, 128, 128, "bf16",
             "softplus0", "sigmoid", "normal0.02"),
    Workload("stream-3frame x20 B1 T10560 H16 D128", 1, 10560, 16, 128, 128, "bf16",
             "softplus0", "sigmoid", "zero", calls=20),
    Workload("cfg-batch B4 T10560 H20 D64 fast-forget", 4, 10560, 20, 64, 64, "bf16",
             "softplus2", "sigmoid", "normal0.02"),
    Workload("long-12frame B1 T42240 H32 D128", 1, 42240, 32, 128, 128, "bf16",
             "uniform0.5", "uniform", "normal0.02"),
)


def f32_to_bf16_bits(x):
    """Round fp32 values to bf16 (round-to-nearest-even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b):
    """Widen bf16 bit patterns to fp32 exactly."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _unit_rows(x):
    n = np.sqrt(np.sum(x * x, axis=-1, keepdims=True, dtype=np.float32))
    return (x / n).astype(np.float32)


def make_inputs(workload, call=0, *, B=None, T=None, H=None, Dk=None, Dv=None,
                dtype=None, state=None, seed=None):
    """Draw one call's inputs for ``workload`` (an index into WORKLOADS or a Workload).

    Keyword overrides change the shape (e.g. a ragged T) while keeping the value
    distributions.  Returns a dict with numpy arrays:
      q, k [B,T,H,Dk] and v [B,T,H,Dv]: float32, or uint16 bf16 bit patterns;
      alpha, beta [B,T,H] float32; state_in [B,H,Dk,Dv] float32 or None;
    plus "dtype" ("f32"/"bf16").
    """
    w = WORKLOADS[workload] if isinstance(workload, int) else workload
    idx = WORKLOADS.index(w) if w in WORKLOADS else 99
    B = w.B if B is None else B
    T = w.T if T is None else T
    H = w.H if H is None else H
    Dk = w.Dk if Dk is None else Dk
    Dv = w.Dv if Dv is None else Dv
    dtype = w.dtype if dtype is None else dtype
    state = w.state if state is None else state
    rng = np.random.default_rng(1000 * idx + call if seed is None else seed)

    q = _unit_rows(rng.standard_normal((B, T, H, Dk), dtype=np.float32))
    k = _unit_rows(rng.standard_normal((B, T, H, Dk), dtype=np.float32))
    v = rng.standard_normal((B, T, H, Dv), dtype=np.float32)
    if w.alpha.startswith("softplus"):
        mu = float(w.alpha[len("softplus"):])
        z = rng.standard_normal((B, T, H)).astype(np.float64) + mu
        alpha = np.exp(-np.logaddexp(0.0, z)).astype(np.float32)
    elif w.alpha == "uniform0.5":
        alpha = rng.uniform(0.5, 1.0, (B, T, H)).astype(np.float32)
    else:
        raise ValueError(w.alpha)
    if w.beta == "sigmoid":
        z = rng.standard_normal((B, T, H)).astype(np.float64)
        beta = (1.0 / (1.0 + np.exp(-z))).astype(np.float32)
    elif w.beta == "uniform":
        beta = rng.uniform(0.0, 1.0, (B, T, H)).astype(np.float32)
    else:
        raise ValueError(w.beta)
    if state == "zero":
        state_in = None
    elif state == "normal0.02":
        state_in = (0.02 * rng.standard_normal((B, H, Dk, Dv), dtype=np.float32)).astype(np.float32)
    else:
        raise ValueError(state)
    if dtype == "bf16":
        q, k, v = f32_to_bf16_bits(q), f32_to_bf16_bits(k), f32_to_bf16_bits(v)
    elif dtype != "f32":
        raise ValueError(dtype)
    return dict(q=q, k=k, v=v, alpha=alpha, beta=beta, state_in=state_in, dtype=dtype)


def make_frame_inputs(workload, frames, *, frame_tokens=None, call=0, B=None, H=None, Dk=None,
                      Dv=None, dtype=None, state=None, seed=None, features="gauss"):
    """Draw one call's inputs for the frame-wise forward: ``frames`` frames of
    ``frame_tokens`` tokens (default 3520, one 44 x 80 latent frame), with the
    value distributions of ``workload``.  The decay is drawn once per (b, frame,
    h); everything else as in make_inputs, in the same order (q, k, v, the alpha
    noise, the beta noise, state_in).  Returns the dict of make_inputs plus
    "frame_tokens", with alpha of shape [B, F, H].

    features="relu" passes the q and k draws through max(0, .) before the
    per-token L2 normalisation (the paper's non-negative feature maps, which
    the normalized readout needs for positive denominators) and adds
    "z_in" [B, H, Dk], a non-negative normalizer state (|N(0, 0.02)|) when the
    workload carries a state, drawn after state_in.
    """
    w = WORKLOADS[workload] if isinstance(workload, int) else workload
    idx = WORKLOADS.index(w) if w in WORKLOADS else 99
    B = w.B if B is None else B
    H = w.H if H is None else H
    Dk = w.Dk if Dk is None else Dk
    Dv = w.Dv if Dv is None else Dv
    N = 3520 if frame_tokens is None else int(frame_tokens)
    F = int(frames)
    T = F * N
    dtype = w.dtype if dtype is None else dtype
    state = w.state if state is None else state
    rng = np.random.default_rng(500000 + 1000 * idx + call if seed is None else seed)

    if features not in ("gauss", "relu"):
        raise ValueError(features)
    feat = (lambda x: np.maximum(x, 0.0)) if features == "relu" else (lambda x: x)
    q = _unit_rows(feat(rng.standard_normal((B, T, H, Dk), dtype=np.float32)))
    k = _unit_rows(feat(rng.standard_normal((B, T, H, Dk), dtype=np.float32)))
    v = rng.standard_normal((B, T, H, Dv), dtype=np.float32)
    if w.alpha.startswith("softplus"):
        mu = float(w.alpha[len("softplus"):])
        z = rng.standard_normal((B, F, H)).astype(np.float64) + mu
        alpha = np.exp(-np.logaddexp(0.0, z)).astype(np.float32)
    elif w.alpha == "uniform0.5":
        alpha = rng.uniform(0.5, 1.0, (B, F, H)).astype(np.float32)
    else:
        raise ValueError(w.alpha)
    if w.beta == "sigmoid":
        z = rng.standard_normal((B, T, H)).astype(np.float64)
        beta = (1.0 / (1.0 + np.exp(-z))).astype(np.float32)
    elif w.beta == "uniform":
        beta = rng.uniform(0.0, 1.0, (B, T, H)).astype(np.float32)
    else:
        raise ValueError(w.beta)
    if state == "zero":
        state_in = None
    elif state == "normal0.02":
        state_in = (0.02 * rng.standard_normal((B, H, Dk, Dv), dtype=np.float32)).astype(np.float32)
    else:
        raise ValueError(state)
    z_in = None
    if features == "relu" and state_in is not None:
        z_in = np.abs(0.02 * rng.standard_normal((B, H, Dk), dtype=np.float32)).astype(np.float32)
    if dtype == "bf16":
        q, k, v = f32_to_bf16_bits(q), f32_to_bf16_bits(k), f32_to_bf16_bits(v)
    elif dtype != "f32":
        raise ValueError(dtype)
    out = dict(q=q, k=k, v=v, alpha=alpha, beta=beta, state_in=state_in, dtype=dtype,
               frame_tokens=N)
    if features == "relu":
        out["z_in"] = z_in
    return out


def rope_3d_params(Dk, base=10000.0):
    """Frequencies and axes of a fixed 3D RoPE over Dk / 2 channel pairs: a
    quarter of the pairs rotate with the time coordinate and three eighths each
    with the latent row and column; along each axis the pair frequencies run
    geometrically from 1 down towards 1 / base.  Returns (freq float32 [Dk/2],
    axis int32 [Dk/2]).  These are inputs to the operator, not its arithmetic."""
    P = Dk // 2
    nt = P // 4
    ny = (P - nt) // 2
    nx = P - nt - ny
    freq, axis = [], []
    for a, n in ((0, nt), (1, ny), (2, nx)):
        freq += [base ** (-j / n) for j in range(n)]
        axis += [a] * n
    return np.array(freq, dtype=np.float32), np.array(axis, dtype=np.int32)


def make_fused_inputs(workload, frames, *, frame_tokens=None, B=None, H=None, Dk=None, Dv=None,
                      state=None, seed=None, lat_w=80, t0=0, dtype="bf16"):
    """Draw one call's inputs for the fused operator (dtype "bf16": q, k, v,
    gate and W_o rounded to bf16 bit patterns; "f32": kept in fp32): the raw query and
    key projections (N(0, 1) with a per-token scale drawn from [0.2, 5], so the
    RMSNorm has work to do), v, the output gate pre-activation (N(0, 1)), the
    per-head projection W_o (N(0, 1 / Dv)), RMSNorm gains (uniform [0.5, 1.5]),
    the 3D RoPE parameters of rope_3d_params, and the decays, write gates and
    states as make_frame_inputs (z_in >= 0).  Draw order: q, k, their scales,
    v, gate, W_o, gains, alpha noise, beta noise, state_in, z_in."""
    w = WORKLOADS[workload] if isinstance(workload, int) else workload
    idx = WORKLOADS.index(w) if w in WORKLOADS else 99
    B = w.B if B is None else B
    H = w.H if H is None else H
    Dk = w.Dk if Dk is None else Dk
    Dv = w.Dv if Dv is None else Dv
    N = 3520 if frame_tokens is None else int(frame_tokens)
    F = int(frames)
    T = F * N
    state = w.state if state is None else state
    rng = np.random.default_rng(700000 + 1000 * idx if seed is None else seed)
    q = rng.standard_normal((B, T, H, Dk), dtype=np.float32)
    k = rng.standard_normal((B, T, H, Dk), dtype=np.float32)
    q *= rng.uniform(0.2, 5.0, (B, T, H, 1)).astype(np.float32)
    k *= rng.uniform(0.2, 5.0, (B, T, H, 1)).astype(np.float32)
    v = rng.standard_normal((B, T, H, Dv), dtype=np.float32)
    gate = rng.standard_normal((B, T, H, Dv), dtype=np.float32)
    w_o = (rng.standard_normal((H, Dv, Dv), dtype=np.float32) / np.float32(np.sqrt(Dv))).astype(np.float32)
    gain_q = rng.uniform(0.5, 1.5, (H, Dk)).astype(np.float32)
    gain_k = rng.uniform(0.5, 1.5, (H, Dk)).astype(np.float32)
    if w.alpha.startswith("softplus"):
        mu = float(w.alpha[len("softplus"):])
        z = rng.standard_normal((B, F, H)).astype(np.float64) + mu
        alpha = np.exp(-np.logaddexp(0.0, z)).astype(np.float32)
    else:
        alpha = rng.uniform(0.5, 1.0, (B, F, H)).astype(np.float32)
    if w.beta == "sigmoid":
        z = rng.standard_normal((B, T, H)).astype(np.float64)
        beta = (1.0 / (1.0 + np.exp(-z))).astype(np.float32)
    else:
        beta = rng.uniform(0.0, 1.0, (B, T, H)).astype(np.float32)
    state_in = z_in = None
    if state == "normal0.02":
        state_in = (0.02 * rng.standard_normal((B, H, Dk, Dv), dtype=np.float32)).astype(np.float32)
        z_in = np.abs(0.02 * rng.standard_normal((B, H, Dk), dtype=np.float32)).astype(np.float32)
    elif state != "zero":
        raise ValueError(state)
    freq, axis = rope_3d_params(Dk)
    if dtype not in ("bf16", "f32"):
        raise ValueError(dtype)
    bf = f32_to_bf16_bits if dtype == "bf16" else (lambda x: x)
    return dict(q=bf(q), k=bf(k), v=bf(v), gate=bf(gate), w_o=bf(w_o), alpha=alpha, beta=beta,
                state_in=state_in, z_in=z_in, gain_q=gain_q, gain_k=gain_k, rope_freq=freq, rope_axis=axis,
                lat_w=int(lat_w), t0=int(t0), frame_tokens=N, dtype=dtype)


def make_device_inputs(workload, device, call=0, *, seed=None):
    """Draw one call's inputs for ``workload`` directly in device memory, with
    the value distributions and draw order of make_inputs but torch's seeded
    generator on the device (fast enough for the largest workloads, whose host
    draws take tens of seconds).  The values differ from make_inputs'; they
    serve timing, never parity.  Returns a dict of torch tensors (q, k, v in
    bf16 or fp32; alpha, beta, state_in in fp32; state_in None for a zero
    state) plus "dtype"."""
    import torch

    w = WORKLOADS[workload] if isinstance(workload, int) else workload
    idx = WORKLOADS.index(w) if w in WORKLOADS else 99
    gen = torch.Generator(device=device)
    gen.manual_seed(900000 + 1000 * idx + call if seed is None else seed)
    B, T, H, Dk, Dv = w.B, w.T, w.H, w.Dk, w.Dv

    def randn(*shape):
        return torch.randn(shape, generator=gen, device=device, dtype=torch.float32)

    def unit_rows(x):
        return x / torch.sqrt(torch.sum(x * x, dim=-1, keepdim=True))

    q = unit_rows(randn(B, T, H, Dk))
    k = unit_rows(randn(B, T, H, Dk))
    v = randn(B, T, H, Dv)
    if w.alpha.startswith("softplus"):
        mu = float(w.alpha[len("softplus"):])
        alpha = torch.exp(-torch.nn.functional.softplus(randn(B, T, H) + mu))
    elif w.alpha == "uniform0.5":
        alpha = 0.5 + 0.5 * torch.rand((B, T, H), generator=gen, device=device)
    else:
        raise ValueError(w.alpha)
    if w.beta == "sigmoid":
        beta = torch.sigmoid(randn(B, T, H))
    elif w.beta == "uniform":
        beta = torch.rand((B, T, H), generator=gen, device=device)
    else:
        raise ValueError(w.beta)
    state_in = 0.02 * randn(B, H, Dk, Dv) if w.state == "normal0.02" else None
    if w.dtype == "bf16":
        q, k, v = q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)
    return dict(q=q.contiguous(), k=k.contiguous(), v=v.contiguous(), alpha=alpha.contiguous(),
                beta=beta.contiguous(), state_in=state_in, dtype=w.dtype)
