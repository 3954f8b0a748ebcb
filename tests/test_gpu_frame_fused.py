"""GPU parity of the fused frame-wise GDN operator (gdn_frame_forward_fused*
through the C ABI: RMSNorm / ReLU / 3D RoPE prologue on the raw q and k, the
rotated-key KV state and the unrotated-key normalizer, the normalized
readout, the SiLU gate and the per-head projection) against the fp64 oracle.

Error metric as for the other frame-wise tests: max|x - x_ref| / max|x_ref|
per tensor (out, state, normalizer state), bound 2e-2 (bf16 q/k/v/gate/W_o;
the features, the gated readout and every product operand are rounded to
bf16, the sines and cosines are the GPU's fast ones).
"""
import numpy as np
import pytest

import gdn_inputs
import oracle

pytestmark = pytest.mark.gpu

TOL = 2e-2
KEYS = ("q", "k", "v", "gate", "w_o", "alpha", "beta", "gain_q", "gain_k", "rope_freq", "rope_axis",
        "state_in", "z_in")


def torch_mod():
    import torch
    return torch


def dev_tensor(a):
    torch = torch_mod()
    if a is None:
        return None
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host_f64(t):
    torch = torch_mod()
    if t.dtype == torch.bfloat16:
        return gdn_inputs.bf16_bits_to_f32(t.view(torch.int16).cpu().numpy().view(np.uint16)).astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


def rel_err(x, ref):
    return float(np.abs(x - ref).max() / max(np.abs(ref).max(), 1e-30))


def run_gpu(gdn, inp, bidirectional=False, key_scale=None, token_splits=None, t0=None):
    t = {k: dev_tensor(inp[k]) for k in KEYS}
    res = gdn.frame_forward_fused(t["q"], t["k"], t["v"], t["gate"], t["w_o"], t["alpha"], t["beta"], t["gain_q"],
                                  t["gain_k"], t["rope_freq"], t["rope_axis"], t["state_in"], t["z_in"],
                                  frame_tokens=inp["frame_tokens"], lat_w=inp["lat_w"],
                                  t0=inp["t0"] if t0 is None else t0, key_scale=key_scale,
                                  bidirectional=bidirectional, token_splits=token_splits)
    torch_mod().cuda.synchronize()
    return res


def oracle_ref(inp, bidirectional=False, key_scale=None, heads=None, t0=None):
    sl = slice(None) if heads is None else list(heads)
    si = None if inp["state_in"] is None else inp["state_in"][:, sl]
    zi = None if inp["z_in"] is None else inp["z_in"][:, sl]
    return oracle.gdn_frame_forward_fused(
        inp["q"][:, :, sl], inp["k"][:, :, sl], inp["v"][:, :, sl], inp["alpha"][:, :, sl], inp["beta"][:, :, sl],
        inp["gate"][:, :, sl], inp["w_o"][sl], si, zi, frame_tokens=inp["frame_tokens"],
        gain_q=inp["gain_q"][sl], gain_k=inp["gain_k"][sl], rope_freq=inp["rope_freq"],
        rope_axis=inp["rope_axis"], lat_w=inp["lat_w"], t0=inp["t0"] if t0 is None else t0, key_scale=key_scale,
        bidirectional=bidirectional)


def check(gdn, inp, label, bidirectional=False, key_scale=None, token_splits=None, heads=None):
    res = run_gpu(gdn, inp, bidirectional, key_scale, token_splits)
    got = [host_f64(x) for x in res]
    ref = oracle_ref(inp, bidirectional, key_scale, heads)
    if heads is not None:
        hs = list(heads)
        got = [got[0][:, :, hs]] + [g[:, hs] for g in got[1:]]
    errs = [rel_err(g, r) for g, r in zip(got, ref)]
    print(f"[fused parity] {label}: out {errs[0]:.3e}, state {errs[1]:.3e}, z {errs[2]:.3e} (tol {TOL:g})",
          flush=True)
    assert all(np.isfinite(g).all() for g in got)
    assert all(e < TOL for e in errs), (label, errs)
    return res


@pytest.mark.parametrize("bidirectional", [False, True])
@pytest.mark.parametrize("Dk,Dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
@pytest.mark.parametrize("F,N", [(1, 1), (2, 63), (3, 64), (2, 65), (4, 200)])
def test_small_frames_fused(gdn, bidirectional, Dk, Dv, F, N):
    inp = gdn_inputs.make_fused_inputs(1, F, frame_tokens=N, B=2, H=3, Dk=Dk, Dv=Dv, lat_w=7, t0=3,
                                       seed=39100 + F * 1000 + N + Dk + 2 * Dv + bidirectional)
    check(gdn, inp, f"{'bidir ' if bidirectional else ''}Dk{Dk} Dv{Dv} F{F} N{N}", bidirectional)


@pytest.mark.parametrize("splits", [1, 3, 100])
def test_token_splits_fused(gdn, splits):
    inp = gdn_inputs.make_fused_inputs(1, 3, frame_tokens=300, H=2, lat_w=20, seed=39200 + splits)
    check(gdn, inp, f"splits={splits}", token_splits=splits)


@pytest.mark.parametrize("lat_w", [1, 5, 64])
def test_grid_widths_and_zero_states(gdn, lat_w):
    inp = gdn_inputs.make_fused_inputs(0, 3, frame_tokens=130, H=2, Dk=64, Dv=64, state="zero", lat_w=lat_w,
                                       seed=39300 + lat_w)
    assert inp["state_in"] is None and inp["z_in"] is None
    check(gdn, inp, f"lat_w={lat_w} zero states", key_scale=0.3)


def test_streaming_advances_time(gdn):
    """Two calls threading both states in place, the second with t0 advanced by
    the first call's frames, each checked against the oracle run call by call."""
    torch = torch_mod()
    inp = gdn_inputs.make_fused_inputs(1, 4, frame_tokens=150, H=2, lat_w=15, t0=4, seed=39500)
    N = inp["frame_tokens"]
    t = {k: dev_tensor(inp[k]) for k in KEYS}
    state, z = t["state_in"].clone(), t["z_in"].clone()
    si, zi = inp["state_in"], inp["z_in"]
    for c in range(2):
        sl = slice(2 * N * c, 2 * N * (c + 1))
        part = dict(inp, q=inp["q"][:, sl], k=inp["k"][:, sl], v=inp["v"][:, sl], gate=inp["gate"][:, sl],
                    alpha=inp["alpha"][:, 2 * c:2 * c + 2], beta=inp["beta"][:, sl], state_in=si, z_in=zi,
                    t0=4 + 2 * c)
        p = {key: dev_tensor(part[key]) for key in ("q", "k", "v", "gate", "alpha", "beta")}
        out = torch.empty_like(p["v"])
        gdn.frame_forward_fused(p["q"], p["k"], p["v"], p["gate"], t["w_o"], p["alpha"], p["beta"], t["gain_q"],
                                t["gain_k"], t["rope_freq"], t["rope_axis"], state, z, frame_tokens=N, lat_w=15,
                                t0=4 + 2 * c, out=out, state_out=state, z_out=z)
        ro, rs, rz = oracle_ref(part)
        torch.cuda.synchronize()
        errs = rel_err(host_f64(out), ro), rel_err(host_f64(state), rs), rel_err(host_f64(z), rz)
        print(f"[fused parity] streaming call {c}: out {errs[0]:.3e}, state {errs[1]:.3e}, z {errs[2]:.3e}",
              flush=True)
        assert all(e < TOL for e in errs)
        si, zi = rs, rz


def test_profile_stages_fused_matches_call(gdn):
    torch = torch_mod()
    inp = gdn_inputs.make_fused_inputs(1, 3, frame_tokens=400, H=4, lat_w=20, seed=39600)
    t = {k: dev_tensor(inp[k]) for k in KEYS}
    ws = gdn.frame_workspace(t["q"], t["v"], 400)
    out = torch.empty_like(t["v"])
    st = torch.empty_like(t["state_in"])
    zo = torch.empty_like(t["z_in"])
    ms = gdn.gdn_frame_profile_stages_fused(t["q"], t["k"], t["v"], t["gate"], t["w_o"], t["alpha"], t["beta"],
                                            t["gain_q"], t["gain_k"], t["rope_freq"], t["rope_axis"],
                                            t["state_in"], t["z_in"], out, st, zo, ws, 400, 20, reps=3)
    assert len(ms) == 4 and all(x > 0 for x in ms), ms
    o2, s2, z2 = run_gpu(gdn, inp, token_splits=0)
    assert torch.equal(out, o2) and torch.equal(st, s2) and torch.equal(zo, z2)


@pytest.mark.parametrize("bidirectional", [False, True])
def test_three_frame_call_fused_full(gdn, bidirectional):
    """The paper's streaming call shape (B1 F3 N3520 on a 44 x 80 latent grid,
    H16 Dk=Dv=128, bf16): every output and both states against the oracle."""
    inp = gdn_inputs.make_fused_inputs(2, 3, state="normal0.02", lat_w=80, t0=6, seed=39900 + bidirectional)
    check(gdn, inp, f"{'bidir ' if bidirectional else ''}B1 F3 N3520 H16 D128", bidirectional)


def test_cfg_batch_fused_sampled_heads(gdn):
    inp = gdn_inputs.make_fused_inputs(3, 3, lat_w=80, seed=39950)
    check(gdn, inp, "B4 F3 N3520 H20 D64 heads 0,7,19", heads=(0, 7, 19))


@pytest.mark.parametrize("N,splits", [(63, 0), (200, 0), (200, 2), (130, 1)])
def test_fused_short_splits_deterministic(gdn, N, splits):
    """Splits of one or two 64-token blocks (fewer than the copy ring holds):
    the copies issued past a split's last block must not land in the slot
    whose keys are being turned into features, so repeated calls agree bitwise
    and with the oracle."""
    torch = torch_mod()
    inp = gdn_inputs.make_fused_inputs(1, 2, frame_tokens=N, B=2, H=3, Dv=64, lat_w=7, seed=39700 + N + splits)
    first = check(gdn, inp, f"Dk128 Dv64 N{N} splits={splits}", token_splits=splits)
    for _ in range(3):
        again = run_gpu(gdn, inp, token_splits=splits)
        assert all(torch.equal(a, b) for a, b in zip(first, again))


@pytest.mark.parametrize("bidirectional", [False, True])
def test_many_frames_fused(gdn, bidirectional):
    """33 frames of 30 tokens on a 6-wide latent grid, time coordinate from 100."""
    inp = gdn_inputs.make_fused_inputs(1, 33, frame_tokens=30, H=2, lat_w=6, t0=100,
                                       seed=39990 + bidirectional)
    check(gdn, inp, f"{'bidir ' if bidirectional else ''}F33 N30", bidirectional)


@pytest.mark.parametrize("bidirectional", [False, True])
@pytest.mark.parametrize("Dk", [64, 128])
def test_write_gates_outside_unit_interval_fused(gdn, Dk, bidirectional):
    """Write gates outside [0, 1] (the interface takes any finite beta): about
    a tenth of the tokens negative and a twentieth above one, with tokens
    64 .. 191 of every frame kept non-negative so that whole 64-token blocks
    have no negative gate and others have some."""
    inp = gdn_inputs.make_fused_inputs(1, 3, frame_tokens=300, H=2, Dk=Dk, Dv=Dk, lat_w=20,
                                       seed=39800 + Dk + bidirectional)
    rng = np.random.default_rng(39850 + Dk + bidirectional)
    b = inp["beta"]
    neg = rng.random(b.shape) < 0.1
    neg.reshape(b.shape[0], 3, 300, b.shape[2])[:, :, 64:192] = False
    b = np.where(neg, -b, b)
    b = np.where(rng.random(b.shape) < 0.05, 3.0 * b, b)
    inp["beta"] = b.astype(np.float32)
    check(gdn, inp, f"{'bidir ' if bidirectional else ''}Dk{Dk} beta in (-1, 3)", bidirectional)


@pytest.mark.parametrize("t0", [5000, 20000])
def test_long_time_coordinate_fused(gdn, t0):
    """Time coordinates whose angles run to thousands of turns (the first time
    pair turns once per 2 pi frames): the kernels reduce each angle to one turn
    before the hardware sine and cosine."""
    inp = gdn_inputs.make_fused_inputs(1, 3, frame_tokens=100, H=2, lat_w=10, t0=t0, seed=39700 + t0 % 97)
    check(gdn, inp, f"t0={t0} F3 N100")
