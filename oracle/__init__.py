"""fp64 CPU oracle for the gated delta-rule forward -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the HIP library
and the product path never calls it.

* :func:`gdn_forward` -- the token-by-token recurrence in fp64 (C library,
  ``gdn_oracle.c``), the reference every GPU result is compared with.
* :mod:`oracle.chunked` -- the chunked (WY / UT) rewrite in fp64 numpy, used
  only to pin the recurrence against an independent algebraic form.
* :mod:`oracle.framewise` -- the paper's frame-wise compact update written as
  printed, used to tie the recurrences to the paper's own equation.
* :func:`gdn_frame_forward` -- the frame-wise recurrence (one decay per frame,
  the frame's tokens writing at once, rescaled keys) in fp64 (C library), the
  reference for the GPU frame-wise path; with ``normalized=True`` also the
  normalizer state and the normalized readout.
* :func:`gdn_frame_forward_fused` -- the whole GDN operator around the frame
  recurrence: RMSNorm / ReLU / 3D RoPE prologue on q and k, the rotated-key
  KV state and unrotated-key normalizer, the normalized readout and the
  SiLU-gate / per-head projection epilogue (C library).
"""
import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None
_DT_QKV = {np.dtype(np.float32): 0, np.dtype(np.uint16): 1, np.dtype(np.float64): 2}
_DT_GATE = {np.dtype(np.float32): 0, np.dtype(np.float64): 2}


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
        vp, i = ctypes.c_void_p, ctypes.c_int
        lib.gdn_oracle_forward.restype = ctypes.c_int
        lib.gdn_oracle_forward.argtypes = [vp, vp, vp, i, vp, vp, i, vp, i, vp, vp,
                                           i, i, i, i, i, i]
        lib.gdn_oracle_frame_forward.restype = ctypes.c_int
        lib.gdn_oracle_frame_forward.argtypes = [vp, vp, vp, i, vp, vp, i, vp, i, vp, vp,
                                                 i, i, i, i, i, i, ctypes.c_double, i]
        lib.gdn_oracle_frame_forward_ex.restype = ctypes.c_int
        lib.gdn_oracle_frame_forward_ex.argtypes = [vp, vp, vp, i, vp, vp, i, vp, vp, i, vp, vp, vp,
                                                    i, i, i, i, i, i, ctypes.c_double, i, ctypes.c_double,
                                                    i, i]
        dp = ctypes.c_void_p
        lib.gdn_oracle_frame_forward_fused.restype = ctypes.c_int
        lib.gdn_oracle_frame_forward_fused.argtypes = [vp, vp, vp, vp, vp, i, vp, vp, i, vp, vp, i,
                                                       dp, dp, ctypes.c_double, dp, vp, i, i,
                                                       vp, vp, vp, i, i, i, i, i, i,
                                                       ctypes.c_double, ctypes.c_double, i, i]
        lib.gdn_oracle_frame_forward_norm.restype = ctypes.c_int
        lib.gdn_oracle_frame_forward_norm.argtypes = [vp, vp, vp, i, vp, vp, i, vp, vp, i, vp, vp, vp,
                                                      i, i, i, i, i, i, ctypes.c_double, ctypes.c_double, i]
        _LIB = lib
    return _LIB


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def gdn_forward(q, k, v, alpha, beta, state_in=None, nthreads=None,
                want_state=True):
    """Run the fp64 token recurrence.

    q, k: [B, T, H, Dk]; v: [B, T, H, Dv] -- all float32, float64, or uint16
    holding bf16 bit patterns (widened exactly).  alpha, beta: [B, T, H]
    float32/float64.  state_in: [B, H, Dk, Dv] float32/float64 or None (zero).
    Returns (out [B, T, H, Dv] float64, state_out [B, H, Dk, Dv] float64 or None).
    """
    q, k, v = (np.ascontiguousarray(x) for x in (q, k, v))
    if not (q.dtype == k.dtype == v.dtype) or q.dtype not in _DT_QKV:
        raise TypeError(f"q/k/v must share one of {list(_DT_QKV)}; got "
                        f"{q.dtype}, {k.dtype}, {v.dtype}")
    alpha = np.ascontiguousarray(alpha)
    beta = np.ascontiguousarray(beta, dtype=alpha.dtype)
    if alpha.dtype not in _DT_GATE:
        raise TypeError(f"alpha/beta dtype {alpha.dtype} unsupported")
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    if k.shape != (B, T, H, Dk) or v.shape != (B, T, H, Dv):
        raise ValueError("q/k/v shape mismatch")
    if alpha.shape != (B, T, H) or beta.shape != (B, T, H):
        raise ValueError("alpha/beta must be [B, T, H]")
    sdt = 0
    if state_in is not None:
        state_in = np.ascontiguousarray(state_in)
        if state_in.dtype not in _DT_GATE:
            raise TypeError(f"state_in dtype {state_in.dtype} unsupported")
        if state_in.shape != (B, H, Dk, Dv):
            raise ValueError("state_in must be [B, H, Dk, Dv]")
        sdt = _DT_GATE[state_in.dtype]
    out = np.empty((B, T, H, Dv), dtype=np.float64)
    state_out = np.empty((B, H, Dk, Dv), dtype=np.float64) if want_state else None
    if nthreads is None:
        nthreads = os.cpu_count() or 1
    rc = _lib().gdn_oracle_forward(
        _ptr(q), _ptr(k), _ptr(v), _DT_QKV[q.dtype],
        _ptr(alpha), _ptr(beta), _DT_GATE[alpha.dtype],
        _ptr(state_in), sdt, _ptr(out), _ptr(state_out),
        B, H, T, Dk, Dv, int(nthreads))
    if rc != 0:
        raise RuntimeError(f"gdn_oracle_forward failed with {rc}")
    return out, state_out


def gdn_frame_forward(q, k, v, alpha, beta, state_in=None, frame_tokens=1, key_scale=None,
                      nthreads=None, want_state=True, normalized=False, z_in=None, eps=1e-6,
                      bidirectional=False):
    """Run the fp64 frame-wise recurrence.

    q, k: [B, T, H, Dk]; v: [B, T, H, Dv] (float32, float64 or bf16 bits as
    uint16); T = F * frame_tokens.  alpha: [B, F, H] (one decay per frame);
    beta: [B, T, H].  key_scale multiplies every key (None: the paper's
    1 / sqrt(Dk * frame_tokens)).  Returns (out [B, T, H, Dv], state_out).

    normalized=True also carries the normalizer state z ([B, H, Dk], from z_in
    or zero) and divides the readout by z . q + eps (equations
    appendix_gdn_z_update and appendix_gdn_readout); it returns
    (out, state_out, z_out).

    bidirectional=True adds to every readout of frame f the backward history
    of the call: the same frame recurrence run over the later frames
    F-1 .. f+1 from a zero state (Algorithm alg:gdn-kernel, Phase B).  The
    returned states are the forward terminal ones.
    """
    q, k, v = (np.ascontiguousarray(x) for x in (q, k, v))
    if not (q.dtype == k.dtype == v.dtype) or q.dtype not in _DT_QKV:
        raise TypeError("q/k/v dtype mismatch or unsupported")
    alpha = np.ascontiguousarray(alpha)
    beta = np.ascontiguousarray(beta, dtype=alpha.dtype)
    if alpha.dtype not in _DT_GATE:
        raise TypeError(f"alpha/beta dtype {alpha.dtype} unsupported")
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    N = int(frame_tokens)
    if N < 1 or T % N:
        raise ValueError("T must be a whole number of frames")
    F = T // N
    if k.shape != (B, T, H, Dk) or v.shape != (B, T, H, Dv):
        raise ValueError("q/k/v shape mismatch")
    if alpha.shape != (B, F, H) or beta.shape != (B, T, H):
        raise ValueError("alpha must be [B, F, H] and beta [B, T, H]")
    sdt = 0
    if state_in is not None:
        state_in = np.ascontiguousarray(state_in)
        if state_in.dtype not in _DT_GATE or state_in.shape != (B, H, Dk, Dv):
            raise ValueError("state_in must be float32/float64 [B, H, Dk, Dv]")
        sdt = _DT_GATE[state_in.dtype]
    if z_in is not None:
        if not normalized:
            raise ValueError("z_in needs normalized=True")
        z_in = np.ascontiguousarray(z_in)
        if z_in.dtype not in _DT_GATE or z_in.shape != (B, H, Dk):
            raise ValueError("z_in must be float32/float64 [B, H, Dk]")
        if state_in is None:
            sdt = _DT_GATE[z_in.dtype]
        elif z_in.dtype != state_in.dtype:   # one stored type for both states
            state_in = state_in.astype(np.float64)
            z_in = z_in.astype(np.float64)
            sdt = 2
    if key_scale is None:
        key_scale = 1.0 / np.sqrt(Dk * N)
    out = np.empty((B, T, H, Dv), dtype=np.float64)
    state_out = np.empty((B, H, Dk, Dv), dtype=np.float64) if want_state else None
    if nthreads is None:
        nthreads = os.cpu_count() or 1
    if bidirectional:
        z_out = np.empty((B, H, Dk), dtype=np.float64) if (want_state and normalized) else None
        rc = _lib().gdn_oracle_frame_forward_ex(
            _ptr(q), _ptr(k), _ptr(v), _DT_QKV[q.dtype],
            _ptr(alpha), _ptr(beta), _DT_GATE[alpha.dtype],
            _ptr(state_in), _ptr(z_in), sdt, _ptr(out), _ptr(state_out), _ptr(z_out),
            B, H, F, N, Dk, Dv, float(key_scale), 1 if normalized else 0, float(eps), 1, int(nthreads))
        if rc != 0:
            raise RuntimeError(f"gdn_oracle_frame_forward_ex failed with {rc}")
        return (out, state_out, z_out) if normalized else (out, state_out)
    if normalized:
        z_out = np.empty((B, H, Dk), dtype=np.float64) if want_state else None
        rc = _lib().gdn_oracle_frame_forward_norm(
            _ptr(q), _ptr(k), _ptr(v), _DT_QKV[q.dtype],
            _ptr(alpha), _ptr(beta), _DT_GATE[alpha.dtype],
            _ptr(state_in), _ptr(z_in), sdt, _ptr(out), _ptr(state_out), _ptr(z_out),
            B, H, F, N, Dk, Dv, float(key_scale), float(eps), int(nthreads))
        if rc != 0:
            raise RuntimeError(f"gdn_oracle_frame_forward_norm failed with {rc}")
        return out, state_out, z_out
    rc = _lib().gdn_oracle_frame_forward(
        _ptr(q), _ptr(k), _ptr(v), _DT_QKV[q.dtype],
        _ptr(alpha), _ptr(beta), _DT_GATE[alpha.dtype],
        _ptr(state_in), sdt, _ptr(out), _ptr(state_out),
        B, H, F, N, Dk, Dv, float(key_scale), int(nthreads))
    if rc != 0:
        raise RuntimeError(f"gdn_oracle_frame_forward failed with {rc}")
    return out, state_out


def gdn_frame_forward_fused(q_raw, k_raw, v, alpha, beta, gate, w_o, state_in=None, z_in=None, *,
                            frame_tokens, gain_q, gain_k, rope_freq, rope_axis, lat_w, t0=0,
                            rms_eps=1e-6, key_scale=None, eps=1e-6, bidirectional=False, nthreads=None,
                            want_state=True):
    """Run the fp64 fused GDN operator (see gdn_oracle_frame_forward_fused in the C file).

    q_raw, k_raw: [B, T, H, Dk]; v, gate: [B, T, H, Dv]; w_o: [H, Dv, Dv] (all float32,
    float64 or bf16 bits as uint16, one type); alpha [B, F, H], beta [B, T, H];
    state_in [B, H, Dk, Dv] and z_in [B, H, Dk] or None; gain_q, gain_k [H, Dk];
    rope_freq [Dk/2] (radians per coordinate unit) and rope_axis [Dk/2] (0 time,
    1 latent row, 2 latent column); lat_w tokens per latent row; t0 the time
    coordinate of the first frame.  key_scale None means 1 / sqrt(Dk * frame_tokens).
    Returns (out [B, T, H, Dv], state_out, z_out), fp64."""
    arrs = [np.ascontiguousarray(x) for x in (q_raw, k_raw, v, gate, w_o)]
    dt = arrs[0].dtype
    if any(a.dtype != dt for a in arrs) or dt not in _DT_QKV:
        raise TypeError("q_raw/k_raw/v/gate/w_o must share one supported dtype")
    q_raw, k_raw, v, gate, w_o = arrs
    alpha = np.ascontiguousarray(alpha)
    beta = np.ascontiguousarray(beta, dtype=alpha.dtype)
    if alpha.dtype not in _DT_GATE:
        raise TypeError(f"alpha/beta dtype {alpha.dtype} unsupported")
    B, T, H, Dk = q_raw.shape
    Dv = v.shape[-1]
    N = int(frame_tokens)
    if N < 1 or T % N or Dk % 2:
        raise ValueError("T must be a whole number of frames and Dk even")
    F = T // N
    if (k_raw.shape != (B, T, H, Dk) or v.shape != (B, T, H, Dv) or gate.shape != (B, T, H, Dv)
            or w_o.shape != (H, Dv, Dv)):
        raise ValueError("shape mismatch")
    if alpha.shape != (B, F, H) or beta.shape != (B, T, H):
        raise ValueError("alpha must be [B, F, H] and beta [B, T, H]")
    gq = np.ascontiguousarray(gain_q, dtype=np.float64)
    gk = np.ascontiguousarray(gain_k, dtype=np.float64)
    fr = np.ascontiguousarray(rope_freq, dtype=np.float64)
    ax = np.ascontiguousarray(rope_axis, dtype=np.int32)
    if gq.shape != (H, Dk) or gk.shape != (H, Dk) or fr.shape != (Dk // 2,) or ax.shape != (Dk // 2,):
        raise ValueError("gains must be [H, Dk], rope_freq and rope_axis [Dk/2]")
    states = [None if x is None else np.ascontiguousarray(x, dtype=np.float64) for x in (state_in, z_in)]
    state_in, z_in = states
    if state_in is not None and state_in.shape != (B, H, Dk, Dv):
        raise ValueError("state_in must be [B, H, Dk, Dv]")
    if z_in is not None and z_in.shape != (B, H, Dk):
        raise ValueError("z_in must be [B, H, Dk]")
    if key_scale is None:
        key_scale = 1.0 / np.sqrt(Dk * N)
    out = np.empty((B, T, H, Dv), dtype=np.float64)
    state_out = np.empty((B, H, Dk, Dv), dtype=np.float64) if want_state else None
    z_out = np.empty((B, H, Dk), dtype=np.float64) if want_state else None
    if nthreads is None:
        nthreads = os.cpu_count() or 1
    rc = _lib().gdn_oracle_frame_forward_fused(
        _ptr(q_raw), _ptr(k_raw), _ptr(v), _ptr(gate), _ptr(w_o), _DT_QKV[dt],
        _ptr(alpha), _ptr(beta), _DT_GATE[alpha.dtype], _ptr(state_in), _ptr(z_in), 2,
        _ptr(gq), _ptr(gk), float(rms_eps), _ptr(fr), _ptr(ax), int(lat_w), int(t0),
        _ptr(out), _ptr(state_out), _ptr(z_out), B, H, F, N, Dk, Dv, float(key_scale), float(eps),
        1 if bidirectional else 0, int(nthreads))
    if rc != 0:
        raise RuntimeError(f"gdn_oracle_frame_forward_fused failed with {rc}")
    return out, state_out, z_out
