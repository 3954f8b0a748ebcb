"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test names the mistake in the oracle it would catch.  None of them
re-types the oracle's loop: they use closed forms, invariants, the paper's own
printed (compact, frame-wise) equation, an independent chunked rewrite, and a
hand-worked example.
"""
import json
import os

import numpy as np
import pytest

import gdn_inputs
import oracle
from oracle.chunked import gdn_chunked
from oracle.framewise import framewise_forward, framewise_forward_normalized

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
rng = np.random.default_rng


def unit_rows(x):
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def rand_case(seed, B=1, T=40, H=2, Dk=8, Dv=6, state=True):
    r = rng(seed)
    q = r.standard_normal((B, T, H, Dk))
    k = unit_rows(r.standard_normal((B, T, H, Dk)))
    v = r.standard_normal((B, T, H, Dv))
    a = r.uniform(0.2, 1.0, (B, T, H))
    b = r.uniform(0.0, 1.0, (B, T, H))
    s = r.standard_normal((B, H, Dk, Dv)) if state else None
    return q, k, v, a, b, s


def rel(x, y):
    return np.abs(x - y).max() / max(np.abs(y).max(), 1e-300)


# P1 -- beta = 0, alpha = 1 leaves the state unchanged (spec invariant).
# Catches: a write that does not scale by beta, a decay applied when alpha = 1.
def test_p1_beta0_alpha1_state_unchanged():
    q, k, v, a, b, s = rand_case(1)
    a[:] = 1.0
    b[:] = 0.0
    out, st = oracle.gdn_forward(q, k, v, a, b, s)
    assert np.array_equal(st, s)
    ref = np.einsum("bthi,bhij->bthj", q, s)
    assert rel(out, ref) < 1e-14


# P2 -- beta = 1, alpha = 1 and a unit key: the state maps k_t to v_t exactly
# (spec invariant).  With q_t = k_t the output is v_t.
# Catches: a sign error in the residual, reading the output before the update,
# a transposed state (Dk != Dv here), a missing k k^T projection.
def test_p2_beta1_alpha1_writes_v():
    q, k, v, a, b, s = rand_case(2, Dk=8, Dv=5)
    a[:] = 1.0
    b[:] = 1.0
    out, st = oracle.gdn_forward(k, k, v, a, b, s)
    assert rel(out, v) < 1e-12
    last = np.einsum("bhij,bhi->bhj", st, k[:, -1])
    assert rel(last, v[:, -1]) < 1e-12


# P3 -- alpha_t* = 0 resets: H_t* = beta k v^T and nothing before t* (state or
# tokens) reaches later outputs (spec invariant).
# Catches: a decay that misses the prediction term (v - p instead of v - alpha p).
def test_p3_alpha0_resets():
    q, k, v, a, b, s = rand_case(3, T=30)
    ts = 17
    a[:, ts] = 0.0
    out1, st1 = oracle.gdn_forward(q[:, :ts + 1], k[:, :ts + 1], v[:, :ts + 1],
                                   a[:, :ts + 1], b[:, :ts + 1], s)
    outer = b[:, ts, :, None, None] * k[:, ts, :, :, None] * v[:, ts, :, None, :]
    assert rel(st1, outer) < 1e-15
    q2, k2, v2, _, b2, s2 = rand_case(33, T=30)
    q2[:, ts:], k2[:, ts:], v2[:, ts:], b2[:, ts:] = q[:, ts:], k[:, ts:], v[:, ts:], b[:, ts:]
    out_a, st_a = oracle.gdn_forward(q, k, v, a, b, s)
    out_b, st_b = oracle.gdn_forward(q2, k2, v2, a, b2, s2)
    assert np.array_equal(out_a[:, ts:], out_b[:, ts:])
    assert np.array_equal(st_a, st_b)


# P4 -- the chunked (WY/UT) rewrite equals the recurrence for every chunk size,
# including a ragged last chunk (spec invariant).
# Catches: any error that the independent chunked algebra does not share.
@pytest.mark.parametrize("chunk", [1, 7, 16, 64, 203])
def test_p4_chunked_equals_recurrence(chunk):
    q, k, v, a, b, s = rand_case(4, B=2, T=203, H=2, Dk=16, Dv=12)
    out, st = oracle.gdn_forward(q, k, v, a, b, s)
    oc, sc = gdn_chunked(q, k, v, a, b, s, chunk=chunk)
    assert rel(oc, out) < 1e-12
    assert rel(sc, st) < 1e-12


def test_p4_chunked_equals_recurrence_workload0():
    inp = gdn_inputs.make_inputs(0)
    out, st = oracle.gdn_forward(inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"])
    oc, sc = gdn_chunked(inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"], chunk=64)
    assert rel(oc, out) < 1e-12 and rel(sc, st) < 1e-12


# P5 -- linearity in (state_in, v) for fixed q, k, alpha, beta.
# Catches: a term that mixes v and the state non-linearly or drops one of them.
def test_p5_linearity():
    q, k, v, a, b, s = rand_case(5)
    o1, s1 = oracle.gdn_forward(q, k, v, a, b, s)
    o2, s2 = oracle.gdn_forward(q, k, np.zeros_like(v), a, b, s)
    o3, s3 = oracle.gdn_forward(q, k, v, a, b, None)
    assert rel(o2 + o3, o1) < 1e-12
    assert rel(s2 + s3, s1) < 1e-12


# P6 -- streaming split: two calls with the state threaded equal one call
# (the streaming cache carries only the terminal state).
# Catches: a state written before the last token, or state_in ignored.
@pytest.mark.parametrize("m", [1, 13, 39])
def test_p6_streaming_split(m):
    q, k, v, a, b, s = rand_case(6)
    o, st = oracle.gdn_forward(q, k, v, a, b, s)
    oa, sa = oracle.gdn_forward(q[:, :m], k[:, :m], v[:, :m], a[:, :m], b[:, :m], s)
    ob, sb = oracle.gdn_forward(q[:, m:], k[:, m:], v[:, m:], a[:, m:], b[:, m:], sa)
    assert np.array_equal(np.concatenate([oa, ob], axis=1), o)
    assert np.array_equal(sb, st)


# P7 -- alpha = 1, beta = 2, v = 0 and unit keys make each step a Householder
# reflection I - 2 k k^T, which preserves the Frobenius norm.
# Catches: a wrong factor on the k k^T term (beta/2, beta^2, ...).
def test_p7_reflection_preserves_norm():
    q, k, v, a, b, s = rand_case(7, T=60)
    a[:] = 1.0
    b[:] = 2.0
    _, st = oracle.gdn_forward(q, k, np.zeros_like(v), a, b, s)
    n0 = np.linalg.norm(s.reshape(s.shape[0], s.shape[1], -1), axis=-1)
    n1 = np.linalg.norm(st.reshape(st.shape[0], st.shape[1], -1), axis=-1)
    assert rel(n1, n0) < 1e-12
    assert rel(st, s) > 1e-3  # the state did move


# P8 -- keys drawn from an orthonormal basis R: in that basis the state rows
# c_j = H^T R[:, j] evolve independently: every row decays by alpha_t and the
# written row becomes alpha_t (1 - beta_t) c_j + beta_t v_t.
# Catches: alpha applied to the write only, beta misplaced, transposed state.
def test_p8_orthonormal_keys_closed_form():
    r = rng(8)
    Dk, Dv, T = 6, 4, 50
    R, _ = np.linalg.qr(r.standard_normal((Dk, Dk)))
    js = r.integers(0, Dk, T)
    k = R[:, js].T[None, :, None, :].copy()
    q = r.standard_normal((1, T, 1, Dk))
    v = r.standard_normal((1, T, 1, Dv))
    a = r.uniform(0.3, 1.0, (1, T, 1))
    b = r.uniform(0.0, 1.0, (1, T, 1))
    H0 = r.standard_normal((1, 1, Dk, Dv))
    out, st = oracle.gdn_forward(q, k, v, a, b, H0)
    C = R.T @ H0[0, 0]
    exp_out = np.zeros((T, Dv))
    for t in range(T):
        j = js[t]
        C = a[0, t, 0] * C
        C[j] = (1.0 - b[0, t, 0]) * C[j] + b[0, t, 0] * v[0, t, 0]
        exp_out[t] = C.T @ (R.T @ q[0, t, 0])
    assert rel(out[0, :, 0], exp_out) < 1e-12
    assert rel(st[0, 0], R @ C) < 1e-12


# P9 -- Dk = Dv = 1: h_T = prod(m) h_0 + sum_t prod_{u>t}(m_u) beta_t k_t v_t with
# m_t = alpha_t (1 - beta_t k_t^2), summed in closed form rather than stepped.
# Catches: a misplaced alpha or beta in the scalar gain / write terms.
def test_p9_scalar_closed_form():
    r = rng(9)
    T = 50
    q = r.standard_normal((1, T, 1, 1))
    k = r.uniform(-1.2, 1.2, (1, T, 1, 1))
    v = r.standard_normal((1, T, 1, 1))
    a = r.uniform(0.5, 1.0, (1, T, 1))
    b = r.uniform(0.0, 1.0, (1, T, 1))
    h0 = r.standard_normal((1, 1, 1, 1))
    out, st = oracle.gdn_forward(q, k, v, a, b, h0)
    m = a[0, :, 0] * (1.0 - b[0, :, 0] * k[0, :, 0, 0] ** 2)
    w = b[0, :, 0] * k[0, :, 0, 0] * v[0, :, 0, 0]
    for t in (0, 1, 24, T - 1):
        h = np.prod(m[:t + 1]) * h0[0, 0, 0, 0] + sum(np.prod(m[s + 1:t + 1]) * w[s] for s in range(t + 1))
        assert abs(out[0, t, 0, 0] - h * q[0, t, 0, 0]) < 1e-12 * max(1.0, abs(h))
        if t == T - 1:
            assert abs(st[0, 0, 0, 0] - h) < 1e-12 * max(1.0, abs(h))


# P10 -- T = 1: H_1 = alpha (I - beta k k^T) H_0 + beta k v^T, as one matrix expression.
def test_p10_single_token():
    q, k, v, a, b, s = rand_case(10, T=1, H=1)
    out, st = oracle.gdn_forward(q, k, v, a, b, s)
    kk, vv, qq = k[0, 0, 0], v[0, 0, 0], q[0, 0, 0]
    H1 = a[0, 0, 0] * (np.eye(len(kk)) - b[0, 0, 0] * np.outer(kk, kk)) @ s[0, 0] + b[0, 0, 0] * np.outer(kk, vv)
    assert rel(st[0, 0], H1) < 1e-14
    assert rel(out[0, 0, 0], H1.T @ qq) < 1e-14


# P11 -- the paper's compact frame-wise equation with one token per frame equals
# the oracle (ties the oracle to the printed equation and orientation S = H^T).
def test_p11_paper_compact_equation_n1():
    q, k, v, a, b, s = rand_case(11, H=1, Dk=7, Dv=5)
    out, st = oracle.gdn_forward(q, k, v, a, b, s)
    Y, S = framewise_forward(q[0, :, 0], k[0, :, 0], v[0, :, 0], a[0, :, 0], b[0, :, 0],
                             S0=s[0, 0].T, N=1)
    assert rel(out[0, :, 0], Y) < 1e-12
    assert rel(st[0, 0], S.T) < 1e-12


# P12 -- a hand-worked two-token example (tests/golden/hand_T2_D2.json).
def test_p12_hand_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "hand_T2_D2.json")))
    shp = lambda x, *d: np.asarray(x, dtype=np.float64).reshape(*d)
    B, T, H, Dk, Dv = g["B"], g["T"], g["H"], g["Dk"], g["Dv"]
    out, st = oracle.gdn_forward(shp(g["q"], B, T, H, Dk), shp(g["k"], B, T, H, Dk),
                                 shp(g["v"], B, T, H, Dv), shp(g["alpha"], B, T, H),
                                 shp(g["beta"], B, T, H), shp(g["state_in"], B, H, Dk, Dv))
    assert np.allclose(out.reshape(T, Dv), g["expected_out"], rtol=0, atol=1e-14)
    assert np.allclose(st.reshape(Dk, Dv), g["expected_state"], rtol=0, atol=1e-14)


# Regression record written by tests/golden/make_golden.py from the oracle itself.
def test_oracle_regression_record():
    g = json.load(open(os.path.join(GOLDEN, "oracle_small.json")))
    inp = gdn_inputs.make_inputs(0, seed=g["seed"], state="normal0.02", **g["shape"])
    out, st = oracle.gdn_forward(inp["q"], inp["k"], inp["v"], inp["alpha"], inp["beta"],
                                 inp["state_in"], nthreads=1)
    exp_out = np.array([float.fromhex(x) for x in g["out"]])
    exp_st = np.array([float.fromhex(x) for x in g["state"]])
    assert rel(out.ravel(), exp_out) < 1e-14
    assert rel(st.ravel(), exp_st) < 1e-14


# The bf16 reader widens exactly, and threading does not change any bit.
def test_bf16_widening_and_threads_bitwise():
    inp = gdn_inputs.make_inputs(1, T=70, H=3)
    q, k, v = inp["q"], inp["k"], inp["v"]
    assert q.dtype == np.uint16
    w = lambda x: gdn_inputs.bf16_bits_to_f32(x).astype(np.float64)
    o1, s1 = oracle.gdn_forward(q, k, v, inp["alpha"], inp["beta"], inp["state_in"], nthreads=1)
    o2, s2 = oracle.gdn_forward(w(q), w(k), w(v), inp["alpha"].astype(np.float64),
                                inp["beta"].astype(np.float64),
                                inp["state_in"].astype(np.float64), nthreads=3)
    assert np.array_equal(o1, o2) and np.array_equal(s1, s2)


def test_oracle_rejects_bad_arguments():
    q, k, v, a, b, s = rand_case(12)
    with pytest.raises(ValueError):
        oracle.gdn_forward(q, k, v[:, :-1], a, b, s)
    with pytest.raises(TypeError):
        oracle.gdn_forward(q.astype(np.float32), k, v, a, b, s)


def test_inputs_recipe():
    inp = gdn_inputs.make_inputs(3, T=128, B=2)
    a, b = inp["alpha"], inp["beta"]
    assert a.shape == (2, 128, 20) and inp["q"].shape == (2, 128, 20, 64)
    assert 0.0 < a.min() and a.max() < 1.0 and np.median(a) < 0.2   # fast-forget heads
    assert 0.0 < b.min() and b.max() < 1.0
    qf = gdn_inputs.bf16_bits_to_f32(inp["q"]).astype(np.float64)
    assert np.allclose(np.linalg.norm(qf, axis=-1), 1.0, atol=1e-2)
    a4 = gdn_inputs.make_inputs(4, T=64)["alpha"]
    assert a4.min() >= 0.5 and a4.max() <= 1.0
    assert gdn_inputs.make_inputs(2, T=64)["state_in"] is None
    x = np.array([1.0, 1.00390625, 1.01171875, -3.0e-3], dtype=np.float32)
    # RNE ties: 1+2^-8 rounds to 1 (even), 1+3*2^-8 rounds up to 1+2^-6
    assert list(gdn_inputs.bf16_bits_to_f32(gdn_inputs.f32_to_bf16_bits(x))[:3]) == [1.0, 1.0, 1.015625]


# ---- frame-wise oracle (one decay per frame, the frame's tokens writing at once) ----

def frame_case(seed, B=1, F=3, N=5, H=2, Dk=8, Dv=6, state=True):
    r = rng(seed)
    T = F * N
    q = r.standard_normal((B, T, H, Dk))
    k = r.standard_normal((B, T, H, Dk))
    v = r.standard_normal((B, T, H, Dv))
    a = r.uniform(0.3, 1.0, (B, F, H))
    b = r.uniform(0.0, 1.0, (B, T, H))
    s = r.standard_normal((B, H, Dk, Dv)) if state else None
    return q, k, v, a, b, s


@pytest.mark.parametrize("F,N", [(1, 1), (4, 1), (3, 5), (2, 17), (1, 40)])
def test_f1_frame_oracle_equals_printed_compact_equation(F, N):
    """The paper's compact update S_f = a S (I - K B K^T) + V B K^T written as
    printed (matrix products, column-token orientation) against the oracle's
    residual loop: catches a transposed state, a missing decay on the
    prediction, a per-token instead of per-frame decay, or a readout from the
    old state."""
    q, k, v, a, b, s = frame_case(100 + 7 * F + N, F=F, N=N)
    ks = 0.37
    o, st = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=ks)
    for h in range(q.shape[2]):
        Y, S = framewise_forward(q[0, :, h], ks * k[0, :, h], v[0, :, h], a[0, :, h], b[0, :, h],
                                 s[0, h].T, N=N)
        assert rel(o[0, :, h], Y) < 1e-12
        assert rel(st[0, h], S.T) < 1e-12


def test_f2_one_token_frames_are_the_token_recurrence():
    """With N = 1 and no key rescale the frame-wise update is the token-wise
    one; ties the two oracles together."""
    q, k, v, _, b, s = rand_case(11, T=30)
    a = rng(12).uniform(0.2, 1.0, (1, 30, 2))
    o1, s1 = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=1, key_scale=1.0)
    o2, s2 = oracle.gdn_forward(q, k, v, a, b, s)
    assert rel(o1, o2) < 1e-13 and rel(s1, s2) < 1e-13


def test_f3_tokens_of_a_frame_write_simultaneously():
    """Permuting the tokens inside every frame permutes their outputs and
    leaves the state unchanged (a sequential in-frame update would not)."""
    F, N = 3, 6
    q, k, v, a, b, s = frame_case(13, F=F, N=N)
    perm = np.concatenate([f * N + rng(14 + f).permutation(N) for f in range(F)])
    o1, s1 = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=0.5)
    o2, s2 = oracle.gdn_frame_forward(q[:, perm], k[:, perm], v[:, perm], a, b[:, perm], s,
                                      frame_tokens=N, key_scale=0.5)
    assert rel(o2, o1[:, perm]) < 1e-12 and rel(s2, s1) < 1e-12
    # ... while the token-wise recurrence over the same tokens is order dependent
    at = np.repeat(a, N, axis=1)
    t1 = oracle.gdn_forward(q, k, v, at, b, s)[1]
    t2 = oracle.gdn_forward(q[:, perm], k[:, perm], v[:, perm], at, b[:, perm], s)[1]
    assert rel(t2, t1) > 1e-6


def test_f4_no_write_only_decays():
    """beta = 0: the state is the initial one times the product of the frame
    decays, and every output reads the state of its own frame."""
    F, N = 4, 3
    q, k, v, a, _, s = frame_case(15, F=F, N=N)
    b = np.zeros((1, F * N, 2))
    o, st = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=0.8)
    cum = np.cumprod(a[0], axis=0)                       # [F, H]
    assert rel(st[0], cum[-1][:, None, None] * s[0]) < 1e-14
    for f in range(F):
        for h in range(2):
            ref = q[0, f * N:(f + 1) * N, h] @ (cum[f, h] * s[0, h])
            assert rel(o[0, f * N:(f + 1) * N, h], ref) < 1e-13


@pytest.mark.parametrize("split", [1, 2, 3])
def test_f5_streaming_split_at_frame_boundaries(split):
    """Carrying the terminal state between calls split at a frame boundary is
    the same computation as one call."""
    F, N = 4, 5
    q, k, v, a, b, s = frame_case(16, F=F, N=N)
    o, st = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=0.4)
    m = split * N
    oa, sa = oracle.gdn_frame_forward(q[:, :m], k[:, :m], v[:, :m], a[:, :split], b[:, :m], s,
                                      frame_tokens=N, key_scale=0.4)
    ob, sb = oracle.gdn_frame_forward(q[:, m:], k[:, m:], v[:, m:], a[:, split:], b[:, m:], sa,
                                      frame_tokens=N, key_scale=0.4)
    assert np.array_equal(np.concatenate([oa, ob], axis=1), o) and np.array_equal(sb, st)


def test_f6_frame_summaries_then_scan():
    """The paper's frame-parallel rewrite: per frame P_f = I - K~^T B K~ and
    A_f = K~^T B V, then H_f = a_f P_f H_{f-1} + A_f and Y_f = Q_f H_f."""
    F, N = 3, 7
    q, k, v, a, b, s = frame_case(17, F=F, N=N, Dk=6, Dv=5)
    ks = 1.0 / np.sqrt(6 * N)
    o, st = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N)   # default key scale
    for h in range(2):
        Hs = s[0, h].copy()
        for f in range(F):
            sl = slice(f * N, (f + 1) * N)
            K = ks * k[0, sl, h]
            Bm = np.diag(b[0, sl, h])
            P = np.eye(6) - K.T @ Bm @ K
            A = K.T @ Bm @ v[0, sl, h]
            Hs = a[0, f, h] * P @ Hs + A
            assert rel(o[0, sl, h], q[0, sl, h] @ Hs) < 1e-12
        assert rel(st[0, h], Hs) < 1e-12


def test_f7_frame_oracle_rejects_bad_arguments():
    q, k, v, a, b, s = frame_case(18, F=2, N=4)
    with pytest.raises(ValueError):
        oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=3)      # T not whole frames
    with pytest.raises(ValueError):
        oracle.gdn_frame_forward(q, k, v, b, b, s, frame_tokens=4)      # alpha per token


# ---- normalizer state and normalized readout (frame-wise) ----

def norm_case(seed, B=1, F=3, N=5, H=2, Dk=8, Dv=6, state=True):
    """Non-negative features (the paper's ReLU feature maps), so that the
    denominators z . q are positive."""
    q, k, v, a, b, s = frame_case(seed, B=B, F=F, N=N, H=H, Dk=Dk, Dv=Dv, state=state)
    z = np.abs(rng(seed + 1).standard_normal((B, H, Dk))) if state else None
    return np.abs(q), np.abs(k), v, a, b, s, z


@pytest.mark.parametrize("F,N", [(1, 1), (4, 1), (3, 5), (2, 17)])
def test_n1_normalizer_equals_printed_compact_equation(F, N):
    """The oracle's correction-based z update (appendix_gdn_z_update) and
    divided readout against the printed compact form (appendix_gdn_z_compact,
    appendix_gdn_readout): catches a z decayed after the write, the wrong key,
    a missing beta on the write, or a readout from the old z."""
    q, k, v, a, b, s, z = norm_case(200 + 3 * F + N, F=F, N=N)
    ks, eps = 0.31, 1e-3
    o, st, zo = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=ks,
                                         normalized=True, z_in=z, eps=eps)
    for h in range(q.shape[2]):
        Y, S, zf = framewise_forward_normalized(q[0, :, h], ks * k[0, :, h], v[0, :, h], a[0, :, h],
                                                b[0, :, h], s[0, h].T, z[0, h], N=N, eps=eps)
        assert rel(o[0, :, h], Y) < 1e-12
        assert rel(st[0, h], S.T) < 1e-12
        assert rel(zo[0, h], zf) < 1e-12


def test_n2_normalizer_is_a_value_column_of_ones():
    """z follows the same recurrence as a column of the state whose values are
    all one: running the un-normalized oracle with v' = [v | 1] gives z as the
    last state column and z . q as the last output column, so the normalized
    output is the numerator divided by that column plus eps."""
    F, N = 4, 6
    q, k, v, a, b, s, z = norm_case(21, F=F, N=N)
    ks, eps = 0.45, 1e-6
    o, st, zo = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=ks,
                                         normalized=True, z_in=z, eps=eps)
    v1 = np.concatenate([v, np.ones(v.shape[:-1] + (1,))], axis=-1)
    s1 = np.concatenate([s, z[..., None]], axis=-1)
    o1, st1 = oracle.gdn_frame_forward(q, k, v1, a, b, s1, frame_tokens=N, key_scale=ks)
    assert rel(zo, st1[..., -1]) < 1e-13
    assert rel(st, st1[..., :-1]) < 1e-13
    assert rel(o, o1[..., :-1] / (o1[..., -1:] + eps)) < 1e-12


def test_n3_orthonormal_keys_store_unit_mass():
    """beta = 1, key scale 1 and orthonormal keys inside a frame: the delta
    rule writes the value 1 for every key, so k_n . z_f = 1 for each token n of
    frame f whatever the earlier state (mass conservation)."""
    Dk, N, F = 8, 5, 3
    r = rng(22)
    k = np.zeros((1, F * N, 1, Dk))
    for f in range(F):
        Qm, _ = np.linalg.qr(r.standard_normal((Dk, Dk)))
        k[0, f * N:(f + 1) * N, 0] = Qm[:, :N].T
    q = np.abs(r.standard_normal((1, F * N, 1, Dk)))
    v = r.standard_normal((1, F * N, 1, 4))
    a = r.uniform(0.2, 1.0, (1, F, 1))
    b = np.ones((1, F * N, 1))
    z0 = r.standard_normal((1, 1, Dk))
    for Fc in range(1, F + 1):
        _, _, zf = oracle.gdn_frame_forward(q[:, :Fc * N], k[:, :Fc * N], v[:, :Fc * N], a[:, :Fc],
                                            b[:, :Fc * N], None, frame_tokens=N, key_scale=1.0,
                                            normalized=True, z_in=z0)
        dots = k[0, (Fc - 1) * N:Fc * N, 0] @ zf[0, 0]
        assert np.abs(dots - 1.0).max() < 1e-13


def test_n4_no_write_only_decays_the_normalizer():
    """beta = 0: z_f = (prod of decays) z_0 and the output is the decayed
    numerator over the decayed denominator plus eps."""
    F, N = 3, 4
    q, k, v, a, _, s, z = norm_case(23, F=F, N=N)
    b = np.zeros((1, F * N, 2))
    eps = 1e-2
    o, st, zo = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=0.7,
                                         normalized=True, z_in=z, eps=eps)
    cum = np.cumprod(a[0], axis=0)
    assert rel(zo[0], cum[-1][:, None] * z[0]) < 1e-14
    for f in range(F):
        for h in range(2):
            qq = q[0, f * N:(f + 1) * N, h]
            ref = (qq @ (cum[f, h] * s[0, h])) / (qq @ (cum[f, h] * z[0, h]) + eps)[:, None]
            assert rel(o[0, f * N:(f + 1) * N, h], ref) < 1e-13


def test_n5_streaming_split_carries_both_states():
    F, N = 4, 3
    q, k, v, a, b, s, z = norm_case(24, F=F, N=N)
    o, st, zo = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=0.6,
                                         normalized=True, z_in=z)
    m = 2 * N
    oa, sa, za = oracle.gdn_frame_forward(q[:, :m], k[:, :m], v[:, :m], a[:, :2], b[:, :m], s,
                                          frame_tokens=N, key_scale=0.6, normalized=True, z_in=z)
    ob, sb, zb = oracle.gdn_frame_forward(q[:, m:], k[:, m:], v[:, m:], a[:, 2:], b[:, m:], sa,
                                          frame_tokens=N, key_scale=0.6, normalized=True, z_in=za)
    assert np.array_equal(np.concatenate([oa, ob], axis=1), o)
    assert np.array_equal(sb, st) and np.array_equal(zb, zo)


def test_n6_empty_normalizer_divides_by_eps():
    """No state and no writes: the denominator is exactly eps."""
    F, N = 2, 3
    q, k, v, a, _, s, _ = norm_case(25, F=F, N=N)
    b = np.zeros((1, F * N, 2))
    o, _, zo = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=0.5,
                                        normalized=True, eps=0.25)
    o0, _ = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=0.5)
    assert np.array_equal(zo, np.zeros_like(zo))
    assert rel(o, o0 / 0.25) < 1e-15


# ---- bidirectional (forward scan from the cache + backward scan within the call) ----

@pytest.mark.parametrize("normalized", [False, True])
@pytest.mark.parametrize("F,N", [(1, 4), (2, 3), (4, 5), (5, 1)])
def test_b1_bidirectional_reads_the_sum_of_two_compact_histories(normalized, F, N):
    """Bidirectional readout from the printed compact update alone.  The
    forward history of frame f is the compact update run over frames 0..f from
    the cached state; the backward one is the same update run over the later
    frames F-1, .., f+1 (in that order) from a zero state, each frame keeping
    its own decay.  The frame reads out from the sum of the two (and, when
    normalized, divides by the sum of the two normalizer states).  Catches a
    backward scan that starts from the cache, includes frame f itself, takes
    its neighbour's decay, or a readout from only one of the histories."""
    q, k, v, a, b, s, z = norm_case(300 + 11 * F + N, F=F, N=N)
    ks, eps = 0.4, 1e-3
    res = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=ks, normalized=normalized,
                                   z_in=z if normalized else None, eps=eps, bidirectional=True)
    o, st = res[0], res[1]

    def compact(frames, h, S0, z0):
        """Terminal (S [Dv, Dk], z [Dk]) of the compact update over `frames`."""
        idx = np.concatenate([np.arange(g * N, (g + 1) * N) for g in frames])
        args = (q[0, idx, h], ks * k[0, idx, h], v[0, idx, h], a[0, frames, h], b[0, idx, h], S0)
        if normalized:
            _, S, zz = framewise_forward_normalized(*args, z0=z0, N=N, eps=eps)
            return S, zz
        return framewise_forward(*args, N=N)[1], None

    Dk, Dv = k.shape[-1], v.shape[-1]
    for h in range(q.shape[2]):
        zin = z[0, h] if normalized else None
        for f in range(F):
            Sf, zf = compact(list(range(f + 1)), h, s[0, h].T, zin)
            Sb, zb = (np.zeros((Dv, Dk)), np.zeros(Dk)) if f == F - 1 else \
                compact(list(range(F - 1, f, -1)), h, None, None)
            Qf = q[0, f * N:(f + 1) * N, h].T
            Y = (Sf + Sb) @ Qf
            if normalized:
                Y = Y / ((zf + zb) @ Qf + eps)
            assert rel(o[0, f * N:(f + 1) * N, h], Y.T) < 1e-11
        Sfin, zfin = compact(list(range(F)), h, s[0, h].T, zin)
        assert rel(st[0, h], Sfin.T) < 1e-12
        if normalized:
            assert rel(res[2][0, h], zfin) < 1e-12


def test_b2_backward_history_is_the_reversed_recurrence():
    """The bidirectional output of frame f exceeds the causal one by Q_f Hb_f,
    where Hb_f is the causal oracle's terminal state over the frames
    F-1, .., f+1 taken in that order from a zero state."""
    F, N = 4, 3
    q, k, v, a, b, s = frame_case(31, F=F, N=N)
    ks = 0.5
    ob, sb = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=ks, bidirectional=True)
    of, sf = oracle.gdn_frame_forward(q, k, v, a, b, s, frame_tokens=N, key_scale=ks)
    assert np.array_equal(sb, sf)                      # the cache carries the forward state
    for f in range(F - 1):
        frames = list(range(F - 1, f, -1))
        idx = np.concatenate([np.arange(g * N, (g + 1) * N) for g in frames])
        _, hb = oracle.gdn_frame_forward(q[:, idx], k[:, idx], v[:, idx], a[:, frames], b[:, idx], None,
                                         frame_tokens=N, key_scale=ks)
        sl = slice(f * N, (f + 1) * N)
        for h in range(2):
            assert rel(ob[0, sl, h] - of[0, sl, h], q[0, sl, h] @ hb[0, h]) < 1e-11


@pytest.mark.parametrize("normalized", [False, True])
def test_b3_single_frame_and_last_frame_are_causal(normalized):
    """No later frame: with F = 1 the bidirectional call is the causal one, and
    in general the last frame's outputs are the causal ones (bitwise)."""
    for F in (1, 3):
        q, k, v, a, b, s, z = norm_case(40 + F, F=F, N=4)
        kw = dict(frame_tokens=4, key_scale=0.6, normalized=normalized, z_in=z if normalized else None)
        rb = oracle.gdn_frame_forward(q, k, v, a, b, s, bidirectional=True, **kw)
        rf = oracle.gdn_frame_forward(q, k, v, a, b, s, **kw)
        last = slice((F - 1) * 4, F * 4)
        assert np.array_equal(rb[0][:, last], rf[0][:, last])
        if F == 1:
            assert np.array_equal(rb[0], rf[0])
        for x, y in zip(rb[1:], rf[1:]):
            assert np.array_equal(x, y)


# ---- fused operator: RMSNorm / ReLU / 3D RoPE prologue, two states, gate and projection ----

def silu(x):
    return x / (1.0 + np.exp(-x))


def fused_case(seed, F=3, N=3, H=2, Dk=8, Dv=5):
    r = rng(seed)
    T = F * N
    return dict(q=r.standard_normal((1, T, H, Dk)), k=r.standard_normal((1, T, H, Dk)),
                v=r.standard_normal((1, T, H, Dv)), gate=r.standard_normal((1, T, H, Dv)),
                w_o=r.standard_normal((H, Dv, Dv)), alpha=r.uniform(0.3, 1.0, (1, F, H)),
                beta=r.uniform(0.1, 1.0, (1, T, H)), s=0.3 * r.standard_normal((1, H, Dk, Dv)),
                z=np.abs(0.3 * r.standard_normal((1, H, Dk))), gq=r.uniform(0.5, 1.5, (H, Dk)),
                gk=r.uniform(0.5, 1.5, (H, Dk)), freq=r.uniform(0.1, 1.3, Dk // 2),
                axis=r.integers(0, 3, Dk // 2).astype(np.int32), N=N)


def run_fused(c, **kw):
    args = dict(frame_tokens=c["N"], gain_q=c["gq"], gain_k=c["gk"], rope_freq=c["freq"], rope_axis=c["axis"],
                lat_w=2, t0=5, rms_eps=0.0)
    args.update(kw)
    return oracle.gdn_frame_forward_fused(c["q"], c["k"], c["v"], c["alpha"], c["beta"], c["gate"], c["w_o"],
                                          c["s"], c["z"], **args)


@pytest.mark.parametrize("bidirectional", [False, True])
def test_u1_orthonormal_features_read_back_their_values(bidirectional):
    """Raw keys c e_{2 j(n)} - d e_m (distinct channel pairs j(n) inside a
    frame, any other channel m) with key gain 1/sqrt(Dk) and key scale 1: the
    RMS is taken over both entries and the ReLU drops the negative one, so the
    feature is lambda e_{2 j(n)} with lambda = c / sqrt(c^2 + d^2), whatever
    rotation follows.  With beta = 1 / lambda^2 each frame writes a projector;
    the query equals the key of its own token.  Then every token reads back
    its own value over a denominator of exactly 1 + eps, whatever the states
    and decays:
        out_n = W_o (SiLU(g_n) o v_n) / (1 + eps).
    A rotation applied to one side only, or differently to q and k, a rotated
    key or query on the normalizer path, a missing ReLU or one taken before the
    RMSNorm, the gate after the projection or a transposed W_o all break it.
    (Bidirectional: the last frame only.)"""
    F, N, H, Dk, Dv = 3, 3, 2, 8, 5
    c = fused_case(61, F=F, N=N, H=H, Dk=Dk, Dv=Dv)
    r = rng(62)
    k = np.zeros((1, F * N, H, Dk))
    beta = np.zeros((1, F * N, H))
    for f in range(F):
        for h in range(H):
            pairs = r.permutation(Dk // 2)[:N]
            for n in range(N):
                cc, dd = r.uniform(0.5, 3.0), r.uniform(0.5, 3.0)
                m = (2 * pairs[n] + 1 + 2 * r.integers(0, Dk // 2)) % Dk      # an odd channel: never 2 j(n)
                k[0, f * N + n, h, 2 * pairs[n]] = cc
                k[0, f * N + n, h, m] = -dd
                beta[0, f * N + n, h] = (cc * cc + dd * dd) / (cc * cc)
    c["k"], c["q"] = k, k.copy()
    c["beta"] = beta
    c["gq"] = c["gk"] = np.full((H, Dk), 1.0 / np.sqrt(Dk))
    eps = 1e-3
    o, _, _ = run_fused(c, key_scale=1.0, eps=eps, bidirectional=bidirectional)
    frames = [F - 1] if bidirectional else range(F)
    for f in frames:
        for n in range(N):
            t = f * N + n
            for h in range(H):
                expect = c["w_o"][h] @ (silu(c["gate"][0, t, h]) * c["v"][0, t, h]) / (1.0 + eps)
                assert rel(o[0, t, h], expect) < 1e-12, (f, n, h)


def test_u2_rotation_direction_and_pairing():
    """A key along e_{2i} written in frame 0 and a query e_{2i+1} + e_{2j} read in
    frame 1 (beta = 0, alpha = 1 there, so the states do not change): the
    numerator is v sin(theta_key - theta_query) on pair i, with
    (x_2i, x_2i+1) -> (x_2i cos - x_2i+1 sin, x_2i sin + x_2i+1 cos), and the
    unrotated denominator is 1 + eps."""
    Dk, Dv, N, H = 8, 3, 2, 1
    i, j = 1, 3
    for axis in (0, 1, 2):
        c = fused_case(63 + axis, F=2, N=N, H=H, Dk=Dk, Dv=Dv)
        c["axis"] = np.full(Dk // 2, axis, dtype=np.int32)
        k = np.full((1, 2 * N, H, Dk), 0.0)
        k[0, 0, 0, 2 * i] = 1.0
        k[0, 1, 0, 2 * j] = 1.0
        k[0, 2:, 0, 0] = 1.0                       # frame 1 keys: not written (beta = 0)
        q = np.full((1, 2 * N, H, Dk), 1.0)
        q[0, 3, 0] = 0.0
        q[0, 3, 0, 2 * i + 1] = q[0, 3, 0, 2 * j] = 1.0
        c["k"], c["q"] = k, q
        c["v"][0, 1] = 0.0
        c["beta"] = np.array([[[1.0], [1.0], [0.0], [0.0]]])
        c["alpha"] = np.array([[[0.7], [1.0]]])
        c["gq"] = np.full((H, Dk), np.sqrt(2.0 / Dk))
        c["gk"] = np.full((H, Dk), 1.0 / np.sqrt(Dk))
        c["w_o"] = np.eye(Dv)[None]
        c["s"], c["z"] = None, None
        eps, lat_w, t0 = 1e-3, 2, 5
        o, _, _ = run_fused(c, key_scale=1.0, eps=eps, lat_w=lat_w, t0=t0)

        def theta(f, s):
            coord = (t0 + f, s // lat_w, s % lat_w)[axis]
            return c["freq"][i] * coord
        expect = silu(c["gate"][0, 3, 0]) * c["v"][0, 0, 0] * np.sin(theta(0, 0) - theta(1, 1)) / (1.0 + eps)
        assert rel(o[0, 3, 0], expect) < 1e-12, axis


def test_u3_rmsnorm_is_per_token_scale_free():
    """With rms_eps = 0, scaling each token's raw q and k by its own positive
    factor changes nothing (the normalisation is over the channels of one
    token and head)."""
    c = fused_case(64)
    o1, s1, z1 = run_fused(c)
    r = rng(65)
    c["q"] = c["q"] * r.uniform(0.1, 10.0, c["q"].shape[:3])[..., None]
    c["k"] = c["k"] * r.uniform(0.1, 10.0, c["k"].shape[:3])[..., None]
    o2, s2, z2 = run_fused(c)
    assert rel(o2, o1) < 1e-12 and rel(s2, s1) < 1e-12 and rel(z2, z1) < 1e-12


def test_u4_no_rotation_and_identity_epilogue_reduce_to_the_normalized_oracle():
    """freq = 0, unit gains, raw q and k already non-negative with a mean square
    of 1 per token (so RMSNorm and ReLU return them), W_o = I: out / SiLU(g)
    is the normalized frame-wise oracle's output on the same q, k."""
    c = fused_case(66, F=3, N=4, Dk=8, Dv=6)
    for key in ("q", "k"):
        x = np.abs(c[key])
        c[key] = x / np.sqrt((x * x).mean(axis=-1, keepdims=True))
    c["freq"] = np.zeros_like(c["freq"])
    c["gq"] = c["gk"] = np.ones_like(c["gq"])
    c["w_o"] = np.stack([np.eye(6)] * 2)
    ks, eps = 0.35, 1e-3
    o, st, zo = run_fused(c, key_scale=ks, eps=eps)
    ro, rs, rz = oracle.gdn_frame_forward(c["q"], c["k"], c["v"], c["alpha"], c["beta"], c["s"], frame_tokens=4,
                                          key_scale=ks, normalized=True, z_in=c["z"], eps=eps)
    assert rel(o / silu(c["gate"]), ro) < 1e-11
    assert rel(st, rs) < 1e-12 and rel(zo, rz) < 1e-12


def test_u5_streaming_split_advances_the_time_coordinate():
    """Two calls (the second with t0 advanced by the first call's frames and the
    carried states) equal one call, bitwise."""
    c = fused_case(67, F=4, N=3)
    o, st, zo = run_fused(c, t0=2)
    a = dict(c, q=c["q"][:, :6], k=c["k"][:, :6], v=c["v"][:, :6], gate=c["gate"][:, :6],
             alpha=c["alpha"][:, :2], beta=c["beta"][:, :6])
    oa, sa, za = run_fused(a, t0=2)
    b = dict(c, q=c["q"][:, 6:], k=c["k"][:, 6:], v=c["v"][:, 6:], gate=c["gate"][:, 6:],
             alpha=c["alpha"][:, 2:], beta=c["beta"][:, 6:], s=sa, z=za)
    ob, sb, zb = run_fused(b, t0=4)
    assert np.array_equal(np.concatenate([oa, ob], axis=1), o)
    assert np.array_equal(sb, st) and np.array_equal(zb, zo)
    ob2, _, _ = run_fused(b, t0=5)
    assert not np.allclose(ob2, ob)                 # the time coordinate matters


def test_u6_bidirectional_single_and_last_frame():
    for F in (1, 3):
        c = fused_case(68 + F, F=F, N=3)
        rb = run_fused(c, bidirectional=True)
        rf = run_fused(c)
        last = slice(3 * (F - 1), 3 * F)
        assert np.array_equal(rb[0][:, last], rf[0][:, last])
        assert np.array_equal(rb[1], rf[1]) and np.array_equal(rb[2], rf[2])
        if F == 3:
            assert not np.allclose(rb[0][:, :3], rf[0][:, :3])
