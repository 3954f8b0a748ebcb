"""The paper's frame-wise compact update, written as printed -- TEST INFRASTRUCTURE ONLY.

Section "Frame-wise Gated DeltaNet", equation appendix_gdn_kv_compact, in the
paper's own column-token orientation (S is Dv x Dk, K_f is Dk x N, V_f is
Dv x N, B_f = diag(beta_f)):

    S_f = alpha_f S_{f-1} (I - K_f B_f K_f^T) + V_f B_f K_f^T

and the un-normalized readout Y_f = S_f Q_f (equation appendix_gdn_readout
without the normalizer, gate or projection).  One alpha per frame is shared by
the frame's N tokens and all of them write at once.  With N = 1 this is the
token recurrence; tests use that case to tie the fp64 oracle to the printed
equation.  (No RoPE or key rescale here.)

framewise_forward_normalized adds the normalizer state as printed in
equation appendix_gdn_z_compact,

    S^z_f = alpha_f (I - K_f B_f K_f^T) S^z_{f-1} + K_f B_f 1,

and the normalized readout of equation appendix_gdn_readout,
Y_f = S_f Q_f / ((S^z_f)^T Q_f + eps), the denominator broadcast over the
value channels (no rotary embedding, so the rotated and unrotated queries and
keys coincide).
"""
import numpy as np


def framewise_forward(q, k, v, alpha_f, beta, S0=None, N=1):
    """One (b, h) stream.

    q, k: [T, Dk]; v: [T, Dv]; alpha_f: [T // N] (one per frame); beta: [T];
    S0: [Dv, Dk] or None.  Returns (Y [T, Dv], S_F [Dv, Dk]) in fp64.
    """
    q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
    T, Dk = k.shape
    Dv = v.shape[1]
    if T % N:
        raise ValueError("T must be a whole number of frames")
    S = np.zeros((Dv, Dk)) if S0 is None else np.asarray(S0, dtype=np.float64).copy()
    Y = np.zeros((T, Dv))
    I = np.eye(Dk)
    for f in range(T // N):
        sl = slice(f * N, (f + 1) * N)
        Kf = k[sl].T                        # Dk x N (column-token convention)
        Vf = v[sl].T                        # Dv x N
        Qf = q[sl].T
        Bf = np.diag(np.asarray(beta[sl], dtype=np.float64))
        S = float(alpha_f[f]) * S @ (I - Kf @ Bf @ Kf.T) + Vf @ Bf @ Kf.T
        Y[sl] = (S @ Qf).T
    return Y, S


def framewise_forward_normalized(q, k, v, alpha_f, beta, S0=None, z0=None, N=1, eps=1e-6):
    """One (b, h) stream with the normalizer.  z0: [Dk] or None.
    Returns (Y [T, Dv], S_F [Dv, Dk], z_F [Dk]) in fp64."""
    q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
    T, Dk = k.shape
    Dv = v.shape[1]
    if T % N:
        raise ValueError("T must be a whole number of frames")
    S = np.zeros((Dv, Dk)) if S0 is None else np.asarray(S0, dtype=np.float64).copy()
    z = np.zeros(Dk) if z0 is None else np.asarray(z0, dtype=np.float64).copy()
    Y = np.zeros((T, Dv))
    I = np.eye(Dk)
    ones = np.ones(N)
    for f in range(T // N):
        sl = slice(f * N, (f + 1) * N)
        Kf = k[sl].T
        Vf = v[sl].T
        Qf = q[sl].T
        Bf = np.diag(np.asarray(beta[sl], dtype=np.float64))
        S = float(alpha_f[f]) * S @ (I - Kf @ Bf @ Kf.T) + Vf @ Bf @ Kf.T
        z = float(alpha_f[f]) * (I - Kf @ Bf @ Kf.T) @ z + Kf @ Bf @ ones
        Y[sl] = ((S @ Qf) / (z @ Qf + eps)).T
    return Y, S, z

