"""GPU parity of the fused frame-wise GDN operator in fp32 (the paper's "ieee"
precision mode; gdn_frame_forward_fused_f32* through the C ABI) against the
fp64 fused oracle.

Error metric as for the other frame-wise tests: max|x - x_ref| / max|x_ref|
per tensor (out, state, normalizer state), bound 1e-4: every feature, product
and readout is fp32 (fp32 MFMA products are exact, accumulation in fp32), the
rotation angles are formed in fp64 with accurate sines and cosines.
"""
import numpy as np
import pytest

import gdn_inputs
import oracle

pytestmark = pytest.mark.gpu

TOL = 1e-4
KEYS = ("q", "k", "v", "gate", "w_o", "alpha", "beta", "gain_q", "gain_k", "rope_freq", "rope_axis",
        "state_in", "z_in")


def torch_mod():
    import torch
    return torch


def dev_tensor(a):
    torch = torch_mod()
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host_f64(t):
    return t.cpu().numpy().astype(np.float64)


def rel_err(x, ref):
    return float(np.abs(x - ref).max() / max(np.abs(ref).max(), 1e-30))


def fused_inputs(workload, frames, **kw):
    return gdn_inputs.make_fused_inputs(workload, frames, dtype="f32", **kw)


def run_gpu(gdn, inp, bidirectional=False, key_scale=None, token_splits=None):
    t = {k: dev_tensor(inp[k]) for k in KEYS}
    assert t["q"].dtype == torch_mod().float32
    res = gdn.frame_forward_fused(t["q"], t["k"], t["v"], t["gate"], t["w_o"], t["alpha"], t["beta"], t["gain_q"],
                                  t["gain_k"], t["rope_freq"], t["rope_axis"], t["state_in"], t["z_in"],
                                  frame_tokens=inp["frame_tokens"], lat_w=inp["lat_w"], t0=inp["t0"],
                                  key_scale=key_scale, bidirectional=bidirectional, token_splits=token_splits)
    torch_mod().cuda.synchronize()
    return res


def oracle_ref(inp, bidirectional=False, key_scale=None, heads=None):
    sl = slice(None) if heads is None else list(heads)
    si = None if inp["state_in"] is None else inp["state_in"][:, sl]
    zi = None if inp["z_in"] is None else inp["z_in"][:, sl]
    return oracle.gdn_frame_forward_fused(
        inp["q"][:, :, sl], inp["k"][:, :, sl], inp["v"][:, :, sl], inp["alpha"][:, :, sl], inp["beta"][:, :, sl],
        inp["gate"][:, :, sl], inp["w_o"][sl], si, zi, frame_tokens=inp["frame_tokens"],
        gain_q=inp["gain_q"][sl], gain_k=inp["gain_k"][sl], rope_freq=inp["rope_freq"],
        rope_axis=inp["rope_axis"], lat_w=inp["lat_w"], t0=inp["t0"], key_scale=key_scale,
        bidirectional=bidirectional)


def check(gdn, inp, label, bidirectional=False, key_scale=None, token_splits=None, heads=None):
    res = run_gpu(gdn, inp, bidirectional, key_scale, token_splits)
    got = [host_f64(x) for x in res]
    ref = oracle_ref(inp, bidirectional, key_scale, heads)
    if heads is not None:
        hs = list(heads)
        got = [got[0][:, :, hs]] + [g[:, hs] for g in got[1:]]
    errs = [rel_err(g, r) for g, r in zip(got, ref)]
    print(f"[fused fp32 parity] {label}: out {errs[0]:.3e}, state {errs[1]:.3e}, z {errs[2]:.3e} (tol {TOL:g})",
          flush=True)
    assert all(np.isfinite(g).all() for g in got)
    assert all(e < TOL for e in errs), (label, errs)
    return res


@pytest.mark.parametrize("bidirectional", [False, True])
@pytest.mark.parametrize("Dk,Dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
@pytest.mark.parametrize("F,N", [(1, 1), (2, 63), (3, 64), (2, 65), (4, 200)])
def test_small_frames_fused_f32(gdn, bidirectional, Dk, Dv, F, N):
    inp = fused_inputs(1, F, frame_tokens=N, B=2, H=3, Dk=Dk, Dv=Dv, lat_w=7, t0=3,
                       seed=49100 + F * 1000 + N + Dk + 2 * Dv + bidirectional)
    check(gdn, inp, f"{'bidir ' if bidirectional else ''}Dk{Dk} Dv{Dv} F{F} N{N}", bidirectional)


@pytest.mark.parametrize("splits", [1, 3, 100])
def test_token_splits_fused_f32(gdn, splits):
    inp = fused_inputs(1, 3, frame_tokens=300, H=2, lat_w=20, seed=49200 + splits)
    check(gdn, inp, f"splits={splits}", token_splits=splits)


@pytest.mark.parametrize("lat_w", [1, 5, 64])
def test_grid_widths_and_zero_states_f32(gdn, lat_w):
    inp = fused_inputs(0, 3, frame_tokens=130, H=2, Dk=64, Dv=64, state="zero", lat_w=lat_w, seed=49300 + lat_w)
    assert inp["state_in"] is None and inp["z_in"] is None
    check(gdn, inp, f"lat_w={lat_w} zero states", key_scale=0.3)


def test_streaming_advances_time_f32(gdn):
    """Two calls threading both states in place, the second with t0 advanced by
    the first call's frames, each checked against the oracle run call by call."""
    torch = torch_mod()
    inp = fused_inputs(1, 4, frame_tokens=150, H=2, lat_w=15, t0=4, seed=49500)
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
        print(f"[fused fp32 parity] streaming call {c}: out {errs[0]:.3e}, state {errs[1]:.3e}, z {errs[2]:.3e}",
              flush=True)
        assert all(e < TOL for e in errs)
        si, zi = rs, rz


def test_profile_stages_fused_f32_matches_call(gdn):
    torch = torch_mod()
    inp = fused_inputs(1, 3, frame_tokens=400, H=4, lat_w=20, seed=49600)
    t = {k: dev_tensor(inp[k]) for k in KEYS}
    ws = gdn.fused_workspace(t["q"], t["v"], 400)
    assert ws.numel() > gdn.frame_workspace(t["q"], t["v"], 400).numel()   # feature maps and readout
    out = torch.empty_like(t["v"])
    st = torch.empty_like(t["state_in"])
    zo = torch.empty_like(t["z_in"])
    ms = gdn.gdn_frame_profile_stages_fused(t["q"], t["k"], t["v"], t["gate"], t["w_o"], t["alpha"], t["beta"],
                                            t["gain_q"], t["gain_k"], t["rope_freq"], t["rope_axis"],
                                            t["state_in"], t["z_in"], out, st, zo, ws, 400, 20, reps=3)
    assert len(ms) == 4 and all(x > 0 for x in ms), ms
    o2, s2, z2 = run_gpu(gdn, inp, token_splits=0)
    assert torch.equal(out, o2) and torch.equal(st, s2) and torch.equal(zo, z2)


def test_workspace_too_small_is_rejected_f32(gdn):
    torch = torch_mod()
    inp = fused_inputs(1, 2, frame_tokens=100, H=2, lat_w=10, seed=49650)
    t = {k: dev_tensor(inp[k]) for k in KEYS}
    small = gdn.frame_workspace(t["q"], t["v"], 100)        # lacks the fp32 feature regions
    with pytest.raises(gdn.GdnError):
        gdn.frame_forward_fused(t["q"], t["k"], t["v"], t["gate"], t["w_o"], t["alpha"], t["beta"], t["gain_q"],
                                t["gain_k"], t["rope_freq"], t["rope_axis"], t["state_in"], t["z_in"],
                                frame_tokens=100, lat_w=10, ws=small, token_splits=0)
    torch.cuda.synchronize()


@pytest.mark.parametrize("bidirectional", [False, True])
def test_three_frame_call_fused_f32_full(gdn, bidirectional):
    """The paper's streaming call shape (B1 F3 N3520 on a 44 x 80 latent grid,
    H16 Dk=Dv=128) in fp32: every output and both states against the oracle."""
    inp = fused_inputs(2, 3, state="normal0.02", lat_w=80, t0=6, seed=49900 + bidirectional)
    check(gdn, inp, f"{'bidir ' if bidirectional else ''}B1 F3 N3520 H16 D128", bidirectional)


def test_cfg_batch_fused_f32_sampled_heads(gdn):
    inp = fused_inputs(3, 3, lat_w=80, seed=49950)
    check(gdn, inp, "B4 F3 N3520 H20 D64 heads 0,7,19", heads=(0, 7, 19))


@pytest.mark.parametrize("bidirectional", [False, True])
def test_many_frames_fused_f32(gdn, bidirectional):
    """33 frames of 30 tokens on a 6-wide latent grid, time coordinate from 100."""
    inp = fused_inputs(1, 33, frame_tokens=30, H=2, lat_w=6, t0=100, seed=49990 + bidirectional)
    check(gdn, inp, f"{'bidir ' if bidirectional else ''}F33 N30", bidirectional)


@pytest.mark.parametrize("t0", [5000, 20000])
def test_long_time_coordinate_fused_f32(gdn, t0):
    """Time coordinates whose angles run to thousands of radians: formed and
    reduced in fp64, so the fp32 features keep their precision."""
    inp = fused_inputs(1, 3, frame_tokens=100, H=2, lat_w=10, t0=t0, seed=49700 + t0 % 97)
    check(gdn, inp, f"t0={t0} F3 N100")
