"""Thin ctypes binding of libgdn.so (the C ABI declared in include/gdn.h).

Argument marshalling only: every step of the GDN chunk forward runs in the HIP
kernels behind the C ABI.  PyTorch supplies device memory and the current
stream.  There is no fallback: if libgdn.so is missing or a call fails, this
module raises.
"""
import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgdn.so")
CHUNK = 64

GDN_OK = 0
_lib = None


class GdnError(RuntimeError):
    """A libgdn call returned a negative status."""

    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} failed: {gdn_status_string(status)} (status {status})")


def lib():
    """Load libgdn.so (built in-tree by paper_2605_30409_amd/build.py)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                              "or python paper_2605_30409_amd/build.py")
        L = ctypes.CDLL(LIB_PATH)
        vp, i, sz, f_p = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p
        core = [vp, vp, vp, f_p, f_p, f_p, vp, f_p, i, i, i, i, i, i]
        for name in ("gdn_chunk_forward", "gdn_chunk_forward_f32"):
            fn = getattr(L, name)
            fn.restype, fn.argtypes = i, core + [vp]
        L.gdn_chunk_forward_noalloc.restype, L.gdn_chunk_forward_noalloc.argtypes = i, core + [vp]
        L.gdn_workspace_check.restype = i
        L.gdn_workspace_check.argtypes = [i, i, i, i, i, i, i, i]
        for name in ("gdn_chunk_forward_ws", "gdn_chunk_forward_f32_ws"):
            fn = getattr(L, name)
            fn.restype, fn.argtypes = i, core + [vp, sz, vp]
        L.gdn_workspace_bytes.restype = sz
        L.gdn_workspace_bytes.argtypes = [i, i, i, i, i, i, i]
        L.gdn_workspace_bytes_ex.restype = sz
        L.gdn_workspace_bytes_ex.argtypes = [i, i, i, i, i, i, i, i]
        L.gdn_scan_group_size.restype = i
        L.gdn_scan_group_size.argtypes = [i, i, i, i, i, i, i, i]
        L.gdn_chunk_forward_ex.restype = i
        L.gdn_chunk_forward_ex.argtypes = core + [i, i, vp, sz, vp]
        L.gdn_profile_stages.restype = i
        L.gdn_profile_stages.argtypes = core + [i, i, vp, sz, i, ctypes.POINTER(ctypes.c_float), vp]
        fl = ctypes.c_float
        fcore = [vp, vp, vp, f_p, f_p, f_p, vp, f_p, i, i, i, i, i, i, fl]
        for name in ("gdn_frame_forward", "gdn_frame_forward_f32"):
            fn = getattr(L, name)
            fn.restype, fn.argtypes = i, fcore + [vp]
        L.gdn_frame_token_splits.restype = i
        L.gdn_frame_token_splits.argtypes = [i, i, i, i, i, i, i]
        L.gdn_frame_workspace_bytes.restype = sz
        L.gdn_frame_workspace_bytes.argtypes = [i, i, i, i, i, i, i, i]
        L.gdn_frame_forward_ex.restype = i
        L.gdn_frame_forward_ex.argtypes = fcore + [i, i, vp, sz, vp]
        L.gdn_frame_profile_stages.restype = i
        L.gdn_frame_profile_stages.argtypes = fcore + [i, i, vp, sz, i, ctypes.POINTER(ctypes.c_float), vp]
        ncore = [vp, vp, vp, f_p, f_p, f_p, f_p, vp, f_p, f_p, i, i, i, i, i, i, fl, fl, i]
        L.gdn_frame_forward_norm.restype = i
        L.gdn_frame_forward_norm.argtypes = ncore + [vp]
        L.gdn_frame_forward_norm_ex.restype = i
        L.gdn_frame_forward_norm_ex.argtypes = ncore + [i, vp, sz, vp]
        L.gdn_frame_profile_stages_norm.restype = i
        L.gdn_frame_profile_stages_norm.argtypes = ncore + [i, vp, sz, i, ctypes.POINTER(ctypes.c_float), vp]
        L.gdn_frame_forward_bidir.restype = i
        L.gdn_frame_forward_bidir.argtypes = ncore + [i, vp]
        L.gdn_frame_forward_bidir_ex.restype = i
        L.gdn_frame_forward_bidir_ex.argtypes = ncore + [i, i, vp, sz, vp]
        L.gdn_frame_profile_stages_bidir.restype = i
        L.gdn_frame_profile_stages_bidir.argtypes = ncore + [i, i, vp, sz, i, ctypes.POINTER(ctypes.c_float),
                                                             vp]
        ucore = [vp] * 16 + [i] * 8 + [fl] * 3 + [i]        # 16 pointers, sizes, lat_w, t0, scales, bidir
        L.gdn_frame_forward_fused.restype = i
        L.gdn_frame_forward_fused.argtypes = ucore + [vp]
        L.gdn_frame_forward_fused_ex.restype = i
        L.gdn_frame_forward_fused_ex.argtypes = ucore + [i, vp, sz, vp]
        L.gdn_frame_profile_stages_fused.restype = i
        L.gdn_frame_profile_stages_fused.argtypes = ucore + [i, vp, sz, i, ctypes.POINTER(ctypes.c_float), vp]
        L.gdn_frame_forward_fused_f32.restype = i
        L.gdn_frame_forward_fused_f32.argtypes = ucore + [vp]
        L.gdn_frame_forward_fused_f32_ex.restype = i
        L.gdn_frame_forward_fused_f32_ex.argtypes = ucore + [i, vp, sz, vp]
        L.gdn_frame_profile_stages_fused_f32.restype = i
        L.gdn_frame_profile_stages_fused_f32.argtypes = ucore + [i, vp, sz, i, ctypes.POINTER(ctypes.c_float), vp]
        L.gdn_frame_fused_workspace_bytes.restype = sz
        L.gdn_frame_fused_workspace_bytes.argtypes = [i, i, i, i, i, i, i, i]
        L.gdn_status_string.restype = ctypes.c_char_p
        L.gdn_status_string.argtypes = [i]
        _lib = L
    return _lib


def gdn_status_string(status):
    return lib().gdn_status_string(int(status)).decode()


def gdn_workspace_bytes(B, H, T, Dk, Dv, chunk=CHUNK, is_bf16=True):
    return int(lib().gdn_workspace_bytes(B, H, T, Dk, Dv, chunk, 1 if is_bf16 else 0))


def gdn_workspace_bytes_ex(B, H, T, Dk, Dv, chunk=CHUNK, is_bf16=True, scan_group=0):
    return int(lib().gdn_workspace_bytes_ex(B, H, T, Dk, Dv, chunk, 1 if is_bf16 else 0,
                                            int(scan_group)))


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check(q, k, v, alpha, beta, state_in, out, state_out, frame_tokens=None):
    """Shape/dtype/device/contiguity checks; returns (B, H, T, Dk, Dv, is_bf16).
    With frame_tokens = N, alpha is one decay per frame, [B, T / N, H]."""
    if q.dtype not in (torch.bfloat16, torch.float32):
        raise TypeError(f"q must be bfloat16 or float32, got {q.dtype}")
    for name, t in (("k", k), ("v", v), ("out", out)):
        if t is not None and t.dtype != q.dtype:
            raise TypeError(f"{name} must have dtype {q.dtype}, got {t.dtype}")
    for name, t in (("alpha", alpha), ("beta", beta), ("state_in", state_in), ("state_out", state_out)):
        if t is not None and t.dtype != torch.float32:
            raise TypeError(f"{name} must be float32, got {t.dtype}")
    dev = q.device
    tensors = dict(q=q, k=k, v=v, alpha=alpha, beta=beta, state_in=state_in, out=out, state_out=state_out)
    for name, t in tensors.items():
        if t is None:
            continue
        if t.device != dev or dev.type != "cuda":
            raise ValueError(f"{name} must be on the same GPU as q ({dev}), got {t.device}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if q.dim() != 4:
        raise ValueError("q must be [B, T, H, Dk]")
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    if tuple(k.shape) != (B, T, H, Dk) or tuple(v.shape) != (B, T, H, Dv):
        raise ValueError("k must be [B, T, H, Dk] and v [B, T, H, Dv]")
    if frame_tokens is None:
        if tuple(alpha.shape) != (B, T, H) or tuple(beta.shape) != (B, T, H):
            raise ValueError("alpha and beta must be [B, T, H]")
    else:
        N = int(frame_tokens)
        if N < 1 or T % N:
            raise ValueError("T must be a whole number of frames of frame_tokens tokens")
        if tuple(alpha.shape) != (B, T // N, H) or tuple(beta.shape) != (B, T, H):
            raise ValueError("alpha must be [B, F, H] (one decay per frame) and beta [B, T, H]")
    for name, t in (("state_in", state_in), ("state_out", state_out)):
        if t is not None and tuple(t.shape) != (B, H, Dk, Dv):
            raise ValueError(f"{name} must be [B, H, Dk, Dv]")
    if out is not None and tuple(out.shape) != (B, T, H, Dv):
        raise ValueError("out must be [B, T, H, Dv]")
    return B, H, T, Dk, Dv, q.dtype == torch.bfloat16


def _stream(dev, stream):
    s = torch.cuda.current_stream(dev) if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _call(name, q, k, v, alpha, beta, state_in, out, state_out, chunk, extra, stream):
    B, H, T, Dk, Dv, is_bf16 = _check(q, k, v, alpha, beta, state_in, out, state_out)
    with torch.cuda.device(q.device):
        rc = getattr(lib(), name)(_ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(beta), _ptr(state_in),
                                  _ptr(out), _ptr(state_out), B, H, T, Dk, Dv, int(chunk), *extra,
                                  _stream(q.device, stream))
    if rc != GDN_OK:
        raise GdnError(name, rc)


def gdn_chunk_forward(q, k, v, alpha, beta, state_in, out, state_out, chunk=CHUNK, stream=None):
    """bf16 path with the library-cached workspace (asynchronous on the current stream)."""
    _call("gdn_chunk_forward", q, k, v, alpha, beta, state_in, out, state_out, chunk, (), stream)


def gdn_chunk_forward_f32(q, k, v, alpha, beta, state_in, out, state_out, chunk=CHUNK, stream=None):
    """fp32 path with the library-cached workspace."""
    _call("gdn_chunk_forward_f32", q, k, v, alpha, beta, state_in, out, state_out, chunk, (), stream)


def gdn_chunk_forward_noalloc(q, k, v, alpha, beta, state_in, out, state_out, chunk=CHUNK, stream=None):
    """bf16 path with the library's static device workspace (no allocation)."""
    _call("gdn_chunk_forward_noalloc", q, k, v, alpha, beta, state_in, out, state_out, chunk, (), stream)


def gdn_chunk_forward_ws(q, k, v, alpha, beta, state_in, out, state_out, ws, chunk=CHUNK, stream=None):
    """bf16 path with a caller-owned workspace (a uint8 device tensor)."""
    _call("gdn_chunk_forward_ws", q, k, v, alpha, beta, state_in, out, state_out, chunk,
          (_ptr(ws), ws.numel()), stream)


def gdn_chunk_forward_f32_ws(q, k, v, alpha, beta, state_in, out, state_out, ws, chunk=CHUNK,
                             stream=None):
    """fp32 path with a caller-owned workspace."""
    _call("gdn_chunk_forward_f32_ws", q, k, v, alpha, beta, state_in, out, state_out, chunk,
          (_ptr(ws), ws.numel()), stream)


def gdn_scan_group_size(B, H, T, Dk, Dv, chunk=CHUNK, scan_group=0, is_bf16=True):
    return int(lib().gdn_scan_group_size(B, H, T, Dk, Dv, chunk, 1 if is_bf16 else 0, int(scan_group)))


def gdn_chunk_forward_ex(q, k, v, alpha, beta, state_in, out, state_out, ws, scan_group=0,
                         chunk=CHUNK, stream=None):
    """Either path (selected by q's dtype) with an explicit scan-group size and workspace."""
    is_bf16 = q.dtype == torch.bfloat16
    _call("gdn_chunk_forward_ex", q, k, v, alpha, beta, state_in, out, state_out, chunk,
          (1 if is_bf16 else 0, int(scan_group), _ptr(ws), ws.numel()), stream)


STAGE_NAMES = ("wy", "group_transfer", "group_scan", "chunk_states", "output")


def gdn_profile_stages(q, k, v, alpha, beta, state_in, out, state_out, ws, reps=20, chunk=CHUNK,
                       scan_group=0, stream=None):
    """Mean per-stage durations in ms over `reps` runs, in the order of STAGE_NAMES."""
    is_bf16 = q.dtype == torch.bfloat16
    ms = (ctypes.c_float * len(STAGE_NAMES))()
    _call("gdn_profile_stages", q, k, v, alpha, beta, state_in, out, state_out, chunk,
          (1 if is_bf16 else 0, int(scan_group), _ptr(ws), ws.numel(), int(reps), ms), stream)
    return [float(x) for x in ms]


def workspace(q, v, chunk=CHUNK, scan_group=0):
    """Allocate a workspace tensor sized for inputs shaped like q [B,T,H,Dk] and v [.., Dv]."""
    B, T, H, Dk = q.shape
    n = gdn_workspace_bytes_ex(B, H, T, Dk, v.shape[-1], chunk, q.dtype == torch.bfloat16,
                               scan_group)
    if n == 0:
        raise ValueError("unsupported shape for the GDN chunk forward")
    return torch.empty(n, dtype=torch.uint8, device=q.device)


def forward(q, k, v, alpha, beta, state_in=None, *, out=None, state_out=None, want_state=True,
            ws=None, chunk=CHUNK, scan_group=None, stream=None):
    """GDN chunk forward.  q, k [B,T,H,Dk] and v [B,T,H,Dv] in bf16 or fp32 (on the GPU);
    alpha, beta [B,T,H] fp32; state_in [B,H,Dk,Dv] fp32 or None (zero).  scan_group
    (chunks per scan group, 0 = the library's choice) selects gdn_chunk_forward_ex.
    Returns (out [B,T,H,Dv] like v, state_out [B,H,Dk,Dv] fp32 or None)."""
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    if out is None:
        out = torch.empty((B, T, H, Dv), dtype=q.dtype, device=q.device)
    if state_out is None and want_state:
        state_out = torch.empty((B, H, Dk, Dv), dtype=torch.float32, device=q.device)
    bf = q.dtype == torch.bfloat16
    if scan_group is not None:
        if ws is None:
            ws = workspace(q, v, chunk, scan_group)
        gdn_chunk_forward_ex(q, k, v, alpha, beta, state_in, out, state_out, ws, scan_group,
                             chunk=chunk, stream=stream)
    elif ws is None:
        fn = gdn_chunk_forward if bf else gdn_chunk_forward_f32
        fn(q, k, v, alpha, beta, state_in, out, state_out, chunk=chunk, stream=stream)
    else:
        fn = gdn_chunk_forward_ws if bf else gdn_chunk_forward_f32_ws
        fn(q, k, v, alpha, beta, state_in, out, state_out, ws, chunk=chunk, stream=stream)
    return out, state_out


# ---------------------------------------------------------------------------
# Frame-wise GDN (gdn_frame_* in include/gdn.h): F frames of N tokens, one
# decay per frame, all tokens of a frame written at once, keys multiplied by
# key_scale (default 1 / sqrt(Dk * N)).

FRAME_STAGE_NAMES = ("summaries", "reduce", "scan", "output")


def default_key_scale(Dk, frame_tokens):
    return 1.0 / float(Dk * frame_tokens) ** 0.5


def gdn_frame_token_splits(B, H, F, N, Dk, Dv, token_splits=0):
    return int(lib().gdn_frame_token_splits(B, H, F, N, Dk, Dv, int(token_splits)))


def gdn_frame_workspace_bytes(B, H, F, N, Dk, Dv, is_bf16=True, token_splits=0):
    return int(lib().gdn_frame_workspace_bytes(B, H, F, N, Dk, Dv, 1 if is_bf16 else 0,
                                               int(token_splits)))


def frame_workspace(q, v, frame_tokens, token_splits=0):
    """Workspace tensor for gdn_frame_forward_ex on inputs shaped like q and v."""
    B, T, H, Dk = q.shape
    N = int(frame_tokens)
    n = gdn_frame_workspace_bytes(B, H, T // N, N, Dk, v.shape[-1], q.dtype == torch.bfloat16,
                                  token_splits)
    if n == 0:
        raise ValueError("unsupported shape for the frame-wise GDN forward")
    return torch.empty(n, dtype=torch.uint8, device=q.device)


def fused_workspace(q, v, frame_tokens, token_splits=0):
    """Workspace tensor for gdn_frame_forward_fused_ex / _f32_ex on inputs shaped like q and v
    (the fp32 operator also keeps its feature maps and gated readout there)."""
    B, T, H, Dk = q.shape
    N = int(frame_tokens)
    n = lib().gdn_frame_fused_workspace_bytes(B, H, T // N, N, Dk, v.shape[-1], 1 if q.dtype == torch.bfloat16
                                              else 0, int(token_splits))
    if n == 0:
        raise ValueError("unsupported shape for the fused frame-wise GDN operator")
    return torch.empty(n, dtype=torch.uint8, device=q.device)


def _frame_call(name, q, k, v, alpha, beta, state_in, out, state_out, frame_tokens, key_scale,
                extra, stream):
    B, H, T, Dk, Dv, _ = _check(q, k, v, alpha, beta, state_in, out, state_out, frame_tokens)
    N = int(frame_tokens)
    ks = default_key_scale(Dk, N) if key_scale is None else float(key_scale)
    with torch.cuda.device(q.device):
        rc = getattr(lib(), name)(_ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(beta), _ptr(state_in),
                                  _ptr(out), _ptr(state_out), B, H, T // N, N, Dk, Dv,
                                  ctypes.c_float(ks), *extra, _stream(q.device, stream))
    if rc != GDN_OK:
        raise GdnError(name, rc)


def gdn_frame_forward_ex(q, k, v, alpha, beta, state_in, out, state_out, ws, frame_tokens,
                         key_scale=None, token_splits=0, stream=None):
    """Either element type (q's dtype selects), explicit workspace and token-split count."""
    is_bf16 = q.dtype == torch.bfloat16
    _frame_call("gdn_frame_forward_ex", q, k, v, alpha, beta, state_in, out, state_out, frame_tokens,
                key_scale, (1 if is_bf16 else 0, int(token_splits), _ptr(ws), ws.numel()), stream)


def gdn_frame_profile_stages(q, k, v, alpha, beta, state_in, out, state_out, ws, frame_tokens,
                             key_scale=None, token_splits=0, reps=20, stream=None):
    """Mean per-stage durations in ms over `reps` runs, in the order of FRAME_STAGE_NAMES."""
    is_bf16 = q.dtype == torch.bfloat16
    ms = (ctypes.c_float * len(FRAME_STAGE_NAMES))()
    _frame_call("gdn_frame_profile_stages", q, k, v, alpha, beta, state_in, out, state_out,
                frame_tokens, key_scale,
                (1 if is_bf16 else 0, int(token_splits), _ptr(ws), ws.numel(), int(reps), ms), stream)
    return [float(x) for x in ms]


def frame_forward(q, k, v, alpha, beta, state_in=None, *, frame_tokens, key_scale=None, out=None,
                  state_out=None, want_state=True, ws=None, token_splits=None, stream=None):
    """Frame-wise GDN forward.  q, k [B,T,H,Dk], v [B,T,H,Dv] (bf16 or fp32, on the GPU) with
    T = F * frame_tokens; alpha [B,F,H] and beta [B,T,H] fp32; state_in [B,H,Dk,Dv] fp32 or
    None.  key_scale None means 1 / sqrt(Dk * frame_tokens).  With ws or token_splits given,
    gdn_frame_forward_ex runs; otherwise the library-cached workspace is used.
    Returns (out [B,T,H,Dv] like v, state_out [B,H,Dk,Dv] fp32 or None)."""
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    if out is None:
        out = torch.empty((B, T, H, Dv), dtype=q.dtype, device=q.device)
    if state_out is None and want_state:
        state_out = torch.empty((B, H, Dk, Dv), dtype=torch.float32, device=q.device)
    if ws is not None or token_splits is not None:
        ts = 0 if token_splits is None else int(token_splits)
        if ws is None:
            ws = frame_workspace(q, v, frame_tokens, ts)
        gdn_frame_forward_ex(q, k, v, alpha, beta, state_in, out, state_out, ws, frame_tokens,
                             key_scale, ts, stream)
    else:
        name = "gdn_frame_forward" if q.dtype == torch.bfloat16 else "gdn_frame_forward_f32"
        _frame_call(name, q, k, v, alpha, beta, state_in, out, state_out, frame_tokens, key_scale,
                    (), stream)
    return out, state_out


# ---------------------------------------------------------------------------
# Frame-wise GDN with the normalizer state (gdn_frame_forward_norm*).

def _check_z(z, B, H, Dk, dev, name):
    if z is None:
        return
    if z.dtype != torch.float32 or tuple(z.shape) != (B, H, Dk):
        raise ValueError(f"{name} must be float32 [B, H, Dk]")
    if z.device != dev or not z.is_contiguous():
        raise ValueError(f"{name} must be contiguous on {dev}")


def _norm_call(name, q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out, frame_tokens,
               key_scale, eps, extra, stream):
    B, H, T, Dk, Dv, is_bf16 = _check(q, k, v, alpha, beta, state_in, out, state_out, frame_tokens)
    _check_z(z_in, B, H, Dk, q.device, "z_in")
    _check_z(z_out, B, H, Dk, q.device, "z_out")
    N = int(frame_tokens)
    ks = default_key_scale(Dk, N) if key_scale is None else float(key_scale)
    with torch.cuda.device(q.device):
        rc = getattr(lib(), name)(_ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(beta), _ptr(state_in),
                                  _ptr(z_in), _ptr(out), _ptr(state_out), _ptr(z_out), B, H, T // N, N,
                                  Dk, Dv, ctypes.c_float(ks), ctypes.c_float(eps), 1 if is_bf16 else 0,
                                  *extra, _stream(q.device, stream))
    if rc != GDN_OK:
        raise GdnError(name, rc)


def gdn_frame_profile_stages_norm(q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out, ws,
                                  frame_tokens, key_scale=None, eps=1e-6, token_splits=0, reps=20,
                                  stream=None):
    """Mean per-stage durations in ms of the normalized frame-wise path."""
    ms = (ctypes.c_float * len(FRAME_STAGE_NAMES))()
    _norm_call("gdn_frame_profile_stages_norm", q, k, v, alpha, beta, state_in, z_in, out, state_out,
               z_out, frame_tokens, key_scale, eps,
               (int(token_splits), _ptr(ws), ws.numel(), int(reps), ms), stream)
    return [float(x) for x in ms]


def frame_forward_norm(q, k, v, alpha, beta, state_in=None, z_in=None, *, frame_tokens, key_scale=None,
                       eps=1e-6, out=None, state_out=None, z_out=None, want_state=True, ws=None,
                       token_splits=None, stream=None):
    """Frame-wise GDN forward with the normalizer state z ([B, H, Dk] fp32) and the
    normalized readout out = (H^T q) / (z . q + eps).  Arguments as frame_forward.
    Returns (out, state_out, z_out)."""
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    if out is None:
        out = torch.empty((B, T, H, Dv), dtype=q.dtype, device=q.device)
    if want_state:
        if state_out is None:
            state_out = torch.empty((B, H, Dk, Dv), dtype=torch.float32, device=q.device)
        if z_out is None:
            z_out = torch.empty((B, H, Dk), dtype=torch.float32, device=q.device)
    if ws is not None or token_splits is not None:
        ts = 0 if token_splits is None else int(token_splits)
        if ws is None:
            ws = frame_workspace(q, v, frame_tokens, ts)
        _norm_call("gdn_frame_forward_norm_ex", q, k, v, alpha, beta, state_in, z_in, out, state_out,
                   z_out, frame_tokens, key_scale, eps, (ts, _ptr(ws), ws.numel()), stream)
    else:
        _norm_call("gdn_frame_forward_norm", q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out,
                   frame_tokens, key_scale, eps, (), stream)
    return out, state_out, z_out


# ---------------------------------------------------------------------------
# Bidirectional frame-wise GDN (gdn_frame_forward_bidir*).

def gdn_frame_profile_stages_bidir(q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out, ws,
                                   frame_tokens, key_scale=None, eps=1e-6, normalized=False,
                                   token_splits=0, reps=20, stream=None):
    """Mean per-stage durations in ms of the bidirectional frame-wise path."""
    ms = (ctypes.c_float * len(FRAME_STAGE_NAMES))()
    _norm_call("gdn_frame_profile_stages_bidir", q, k, v, alpha, beta, state_in, z_in, out, state_out,
               z_out, frame_tokens, key_scale, eps,
               (1 if normalized else 0, int(token_splits), _ptr(ws), ws.numel(), int(reps), ms), stream)
    return [float(x) for x in ms]


def frame_forward_bidir(q, k, v, alpha, beta, state_in=None, z_in=None, *, frame_tokens, key_scale=None,
                        normalized=False, eps=1e-6, out=None, state_out=None, z_out=None, want_state=True,
                        ws=None, token_splits=None, stream=None):
    """Bidirectional frame-wise GDN forward: every frame reads out the forward state
    (from state_in) plus the backward history of the call's later frames (from
    zero).  Arguments as frame_forward, and with normalized=True as
    frame_forward_norm (z_in / z_out are ignored otherwise).  The returned states
    are the forward terminal ones.  Returns (out, state_out), or
    (out, state_out, z_out) when normalized."""
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    if not normalized:
        z_in = z_out = None
    if out is None:
        out = torch.empty((B, T, H, Dv), dtype=q.dtype, device=q.device)
    if want_state:
        if state_out is None:
            state_out = torch.empty((B, H, Dk, Dv), dtype=torch.float32, device=q.device)
        if normalized and z_out is None:
            z_out = torch.empty((B, H, Dk), dtype=torch.float32, device=q.device)
    nf = 1 if normalized else 0
    if ws is not None or token_splits is not None:
        ts = 0 if token_splits is None else int(token_splits)
        if ws is None:
            ws = frame_workspace(q, v, frame_tokens, ts)
        _norm_call("gdn_frame_forward_bidir_ex", q, k, v, alpha, beta, state_in, z_in, out, state_out,
                   z_out, frame_tokens, key_scale, eps, (nf, ts, _ptr(ws), ws.numel()), stream)
    else:
        _norm_call("gdn_frame_forward_bidir", q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out,
                   frame_tokens, key_scale, eps, (nf,), stream)
    return (out, state_out, z_out) if normalized else (out, state_out)


# ---------------------------------------------------------------------------
# The fused operator (gdn_frame_forward_fused*): RMSNorm / ReLU / 3D RoPE on the
# raw q and k, the two states, the normalized readout, SiLU gate and W_o.

def _check_param(t, shape, dtype, dev, name):
    if t.dtype != dtype or tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must be {dtype} {list(shape)}")
    if t.device != dev or not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous on {dev}")


def _fused_call(name, q, k, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq, rope_axis, state_in, z_in,
                out, state_out, z_out, frame_tokens, lat_w, t0, key_scale, rms_eps, eps, bidirectional, extra,
                stream):
    B, H, T, Dk, Dv, is_bf16 = _check(q, k, v, alpha, beta, state_in, out, state_out, frame_tokens)
    dev = q.device
    dt = torch.bfloat16 if is_bf16 else torch.float32
    _check_param(gate, v.shape, dt, dev, "gate")
    _check_param(w_o, (H, Dv, Dv), dt, dev, "w_o")
    if not is_bf16:
        name = name.replace("fused", "fused_f32")
    _check_param(gain_q, (H, Dk), torch.float32, dev, "gain_q")
    _check_param(gain_k, (H, Dk), torch.float32, dev, "gain_k")
    _check_param(rope_freq, (Dk // 2,), torch.float32, dev, "rope_freq")
    _check_param(rope_axis, (Dk // 2,), torch.int32, dev, "rope_axis")
    _check_z(z_in, B, H, Dk, dev, "z_in")
    _check_z(z_out, B, H, Dk, dev, "z_out")
    N = int(frame_tokens)
    ks = default_key_scale(Dk, N) if key_scale is None else float(key_scale)
    with torch.cuda.device(dev):
        rc = getattr(lib(), name)(_ptr(q), _ptr(k), _ptr(v), _ptr(gate), _ptr(w_o), _ptr(alpha), _ptr(beta),
                                  _ptr(gain_q), _ptr(gain_k), _ptr(rope_freq), _ptr(rope_axis), _ptr(state_in),
                                  _ptr(z_in), _ptr(out), _ptr(state_out), _ptr(z_out), B, H, T // N, N, Dk, Dv,
                                  int(lat_w), int(t0), ctypes.c_float(ks), ctypes.c_float(rms_eps),
                                  ctypes.c_float(eps), 1 if bidirectional else 0, *extra, _stream(dev, stream))
    if rc != GDN_OK:
        raise GdnError(name, rc)


def gdn_frame_profile_stages_fused(q, k, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq, rope_axis,
                                   state_in, z_in, out, state_out, z_out, ws, frame_tokens, lat_w, t0=0,
                                   key_scale=None, rms_eps=1e-6, eps=1e-6, bidirectional=False, token_splits=0,
                                   reps=20, stream=None):
    """Mean per-stage durations in ms of the fused operator."""
    ms = (ctypes.c_float * len(FRAME_STAGE_NAMES))()
    _fused_call("gdn_frame_profile_stages_fused", q, k, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq,
                rope_axis, state_in, z_in, out, state_out, z_out, frame_tokens, lat_w, t0, key_scale, rms_eps,
                eps, bidirectional, (int(token_splits), _ptr(ws), ws.numel(), int(reps), ms), stream)
    return [float(x) for x in ms]


def frame_forward_fused(q, k, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq, rope_axis, state_in=None,
                        z_in=None, *, frame_tokens, lat_w, t0=0, key_scale=None, rms_eps=1e-6, eps=1e-6,
                        bidirectional=False, out=None, state_out=None, z_out=None, want_state=True, ws=None,
                        token_splits=None, stream=None):
    """The fused frame-wise GDN operator, bf16 or fp32 (all of q, k, v, gate,
    w_o one type; fp32 runs the fp32 mode).  q, k: the raw projections
    [B, T, H, Dk]; v, gate (pre-SiLU) [B, T, H, Dv]; w_o [H, Dv, Dv] (row = output
    channel); alpha [B, F, H], beta [B, T, H] fp32; gain_q, gain_k [H, Dk] fp32
    RMSNorm gains; rope_freq [Dk/2] fp32 and rope_axis [Dk/2] int32 (0 time, 1
    latent row, 2 latent column) of the 3D RoPE, with lat_w tokens per latent row
    and t0 the time coordinate of the first frame; state_in [B, H, Dk, Dv] and
    z_in [B, H, Dk] fp32 or None.  Returns (out [B, T, H, Dv] like q, state_out,
    z_out)."""
    B, T, H, Dk = q.shape
    Dv = v.shape[-1]
    if out is None:
        out = torch.empty((B, T, H, Dv), dtype=q.dtype, device=q.device)
    if want_state:
        if state_out is None:
            state_out = torch.empty((B, H, Dk, Dv), dtype=torch.float32, device=q.device)
        if z_out is None:
            z_out = torch.empty((B, H, Dk), dtype=torch.float32, device=q.device)
    args = (q, k, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq, rope_axis, state_in, z_in, out, state_out,
            z_out, frame_tokens, lat_w, t0, key_scale, rms_eps, eps, bidirectional)
    if ws is not None or token_splits is not None:
        ts = 0 if token_splits is None else int(token_splits)
        if ws is None:
            ws = fused_workspace(q, v, frame_tokens, ts)
        _fused_call("gdn_frame_forward_fused_ex", *args, (ts, _ptr(ws), ws.numel()), stream)
    else:
        _fused_call("gdn_frame_forward_fused", *args, (), stream)
    return out, state_out, z_out
