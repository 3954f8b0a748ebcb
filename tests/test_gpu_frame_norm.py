"""GPU parity of the frame-wise GDN forward with the normalizer state and the
normalized readout (gdn_frame_forward_norm* through the C ABI) against the
fp64 oracle.

Inputs use the paper's non-negative feature maps (ReLU before the per-token
L2 normalisation), so the denominators z . q + eps are positive.  Error
metric and bounds as elsewhere: max|x - x_ref| / max|x_ref| per tensor (out,
state, normalizer state), 1e-4 for the fp32 path and 2e-2 for bf16 q/k/v.
"""
import numpy as np
import pytest

import gdn_inputs
import oracle

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


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


def run_gpu(gdn, inp, key_scale=None, eps=1e-6, token_splits=None):
    t = {k: dev_tensor(inp[k]) for k in ("q", "k", "v", "alpha", "beta", "state_in", "z_in")}
    out, st, zo = gdn.frame_forward_norm(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"],
                                         t["z_in"], frame_tokens=inp["frame_tokens"], key_scale=key_scale,
                                         eps=eps, token_splits=token_splits)
    torch_mod().cuda.synchronize()
    return out, st, zo


def oracle_ref(inp, key_scale=None, eps=1e-6, heads=None):
    sl = slice(None) if heads is None else list(heads)
    si = None if inp["state_in"] is None else inp["state_in"][:, sl]
    zi = None if inp["z_in"] is None else inp["z_in"][:, sl]
    return oracle.gdn_frame_forward(inp["q"][:, :, sl], inp["k"][:, :, sl], inp["v"][:, :, sl],
                                    inp["alpha"][:, :, sl], inp["beta"][:, :, sl], si,
                                    frame_tokens=inp["frame_tokens"], key_scale=key_scale,
                                    normalized=True, z_in=zi, eps=eps)


def check(gdn, inp, label, key_scale=None, eps=1e-6, token_splits=None, heads=None):
    out, st, zo = run_gpu(gdn, inp, key_scale, eps, token_splits)
    o, s, z = host_f64(out), host_f64(st), host_f64(zo)
    ref_o, ref_s, ref_z = oracle_ref(inp, key_scale, eps, heads)
    if heads is not None:
        hs = list(heads)
        o, s, z = o[:, :, hs], s[:, hs], z[:, hs]
    eo, es, ez = rel_err(o, ref_o), rel_err(s, ref_s), rel_err(z, ref_z)
    tol = TOL[inp["dtype"]]
    print(f"[norm parity] {label}: out {eo:.3e}, state {es:.3e}, z {ez:.3e} (tol {tol:g})", flush=True)
    assert np.isfinite(o).all() and np.isfinite(s).all() and np.isfinite(z).all()
    assert eo < tol and es < tol and ez < tol, (label, eo, es, ez)
    return out, st, zo


def relu_inputs(workload, F, N, **kw):
    return gdn_inputs.make_frame_inputs(workload, F, frame_tokens=N, features="relu", **kw)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("Dk,Dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
@pytest.mark.parametrize("F,N", [(1, 1), (3, 1), (2, 63), (3, 64), (2, 65), (4, 200)])
def test_small_frames_normalized(gdn, dtype, Dk, Dv, F, N):
    inp = relu_inputs(1, F, N, B=2, H=3, Dk=Dk, Dv=Dv, dtype=dtype, seed=19100 + F * 1000 + N + Dk + 2 * Dv)
    check(gdn, inp, f"{dtype} Dk{Dk} Dv{Dv} F{F} N{N}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("splits", [1, 3, 100])
def test_token_splits_normalized(gdn, dtype, splits):
    inp = relu_inputs(1, 3, 300, H=2, dtype=dtype, seed=19200 + splits)
    check(gdn, inp, f"{dtype} splits={splits}", token_splits=splits)


def test_zero_states_and_large_eps(gdn):
    inp = relu_inputs(0, 3, 130, H=2, Dk=64, Dv=64, state="zero", seed=19300)
    assert inp["z_in"] is None and inp["state_in"] is None
    check(gdn, inp, "f32 zero states")
    check(gdn, inp, "f32 eps=0.5", eps=0.5, key_scale=0.2)


def test_no_write_divides_decayed_states(gdn):
    """beta = 0: z_F = prod(alpha) z_0, and the output is the decayed numerator
    over the decayed denominator plus eps."""
    inp = relu_inputs(0, 3, 70, H=2, Dk=64, Dv=64, state="normal0.02", seed=19400)
    inp["beta"][:] = 0.0
    _, _, zo = run_gpu(gdn, inp)
    decay = np.prod(inp["alpha"].astype(np.float64), axis=1)
    assert rel_err(host_f64(zo), decay[:, :, None] * inp["z_in"].astype(np.float64)) < 1e-5
    check(gdn, inp, "f32 beta=0")


def test_in_place_states_streaming(gdn):
    """Two calls with state_in == state_out and z_in == z_out equal one call."""
    torch = torch_mod()
    inp = relu_inputs(1, 4, 150, H=2, seed=19500)
    N = inp["frame_tokens"]
    ref_o, ref_s, ref_z = oracle_ref(inp)
    state = dev_tensor(inp["state_in"]).clone()
    z = dev_tensor(inp["z_in"]).clone()
    outs = []
    for c in range(2):
        sl = slice(2 * N * c, 2 * N * (c + 1))
        t = {key: dev_tensor(inp[key][:, sl]) for key in ("q", "k", "v", "beta")}
        al = dev_tensor(inp["alpha"][:, 2 * c:2 * c + 2])
        out = torch.empty_like(t["v"])
        gdn.frame_forward_norm(t["q"], t["k"], t["v"], al, t["beta"], state, z, frame_tokens=N,
                               out=out, state_out=state, z_out=z)
        outs.append(out)
    torch.cuda.synchronize()
    o = np.concatenate([host_f64(x) for x in outs], axis=1)
    eo, es, ez = rel_err(o, ref_o), rel_err(host_f64(state), ref_s), rel_err(host_f64(z), ref_z)
    print(f"[norm parity] streaming in place: out {eo:.3e}, state {es:.3e}, z {ez:.3e}", flush=True)
    assert eo < TOL["bf16"] and es < TOL["bf16"] and ez < TOL["bf16"]


def test_profile_stages_norm_matches_call(gdn):
    torch = torch_mod()
    inp = relu_inputs(1, 3, 400, H=4, seed=19600)
    t = {k: dev_tensor(inp[k]) for k in ("q", "k", "v", "alpha", "beta", "state_in", "z_in")}
    ws = gdn.frame_workspace(t["q"], t["v"], 400)
    out = torch.empty_like(t["v"])
    st = torch.empty_like(t["state_in"])
    zo = torch.empty_like(t["z_in"])
    ms = gdn.gdn_frame_profile_stages_norm(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"],
                                           t["z_in"], out, st, zo, ws, 400, reps=3)
    assert len(ms) == 4 and all(x > 0 for x in ms), ms
    o2, s2, z2 = run_gpu(gdn, inp, token_splits=0)
    assert torch.equal(out, o2) and torch.equal(st, s2) and torch.equal(zo, z2)


def test_three_frame_call_normalized_full(gdn):
    """The paper's streaming call shape (B1 F3 N3520 H16 Dk=Dv=128, bf16), every
    output and both states against the oracle."""
    inp = relu_inputs(2, 3, 3520, state="normal0.02", seed=19900)
    check(gdn, inp, "bf16 B1 F3 N3520 H16 D128")


def test_cfg_batch_normalized_sampled_heads(gdn):
    inp = relu_inputs(3, 3, 3520, seed=19950)
    check(gdn, inp, "bf16 B4 F3 N3520 H20 D64 heads 0,7,19", heads=(0, 7, 19))


def test_many_frames_normalized(gdn):
    inp = relu_inputs(1, 37, 20, H=2, seed=19990)
    check(gdn, inp, "bf16 F37 N20")
