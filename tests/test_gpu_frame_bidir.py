"""GPU parity of the bidirectional frame-wise GDN forward
(gdn_frame_forward_bidir* through the C ABI) against the fp64 oracle, with
and without the normalizer.

Error metric and bounds as for the other frame-wise tests: max|x - x_ref| /
max|x_ref| per tensor, 1e-4 for the fp32 path and 2e-2 for bf16 q/k/v.  The
normalized cases use the non-negative feature maps (ReLU before the per-token
L2 normalisation) so that the denominators stay positive.
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


def make(workload, F, N, normalized, **kw):
    return gdn_inputs.make_frame_inputs(workload, F, frame_tokens=N, features="relu" if normalized else "gauss",
                                        **kw)


def run_gpu(gdn, inp, normalized, key_scale=None, eps=1e-6, token_splits=None):
    t = {k: dev_tensor(inp.get(k)) for k in ("q", "k", "v", "alpha", "beta", "state_in", "z_in")}
    res = gdn.frame_forward_bidir(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"], t["z_in"],
                                  frame_tokens=inp["frame_tokens"], key_scale=key_scale, normalized=normalized,
                                  eps=eps, token_splits=token_splits)
    torch_mod().cuda.synchronize()
    return res


def oracle_ref(inp, normalized, key_scale=None, eps=1e-6, heads=None, bidirectional=True):
    sl = slice(None) if heads is None else list(heads)
    si = None if inp["state_in"] is None else inp["state_in"][:, sl]
    zi = None if inp.get("z_in") is None else inp["z_in"][:, sl]
    return oracle.gdn_frame_forward(inp["q"][:, :, sl], inp["k"][:, :, sl], inp["v"][:, :, sl],
                                    inp["alpha"][:, :, sl], inp["beta"][:, :, sl], si,
                                    frame_tokens=inp["frame_tokens"], key_scale=key_scale,
                                    normalized=normalized, z_in=zi if normalized else None, eps=eps,
                                    bidirectional=bidirectional)


def check(gdn, inp, normalized, label, key_scale=None, eps=1e-6, token_splits=None, heads=None):
    res = run_gpu(gdn, inp, normalized, key_scale, eps, token_splits)
    got = [host_f64(x) for x in res]
    ref = oracle_ref(inp, normalized, key_scale, eps, heads)
    if heads is not None:
        hs = list(heads)
        got = [got[0][:, :, hs]] + [g[:, hs] for g in got[1:]]
    errs = [rel_err(g, r) for g, r in zip(got, ref)]
    tol = TOL[inp["dtype"]]
    print(f"[bidir parity] {label}: " + ", ".join(f"{n} {e:.3e}" for n, e in zip(("out", "state", "z"), errs))
          + f" (tol {tol:g})", flush=True)
    assert all(np.isfinite(g).all() for g in got)
    assert all(e < tol for e in errs), (label, errs)
    return res


@pytest.mark.parametrize("normalized", [False, True])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("Dk,Dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
@pytest.mark.parametrize("F,N", [(1, 1), (2, 1), (3, 63), (2, 65), (5, 64), (4, 200)])
def test_small_frames_bidirectional(gdn, normalized, dtype, Dk, Dv, F, N):
    inp = make(1, F, N, normalized, B=2, H=3, Dk=Dk, Dv=Dv, dtype=dtype,
               seed=29100 + F * 1000 + N + Dk + 2 * Dv + 7 * normalized)
    check(gdn, inp, normalized, f"{'norm ' if normalized else ''}{dtype} Dk{Dk} Dv{Dv} F{F} N{N}")


@pytest.mark.parametrize("normalized", [False, True])
@pytest.mark.parametrize("splits", [1, 3, 100])
def test_token_splits_bidirectional(gdn, normalized, splits):
    inp = make(1, 3, 300, normalized, H=2, dtype="bf16", seed=29200 + splits)
    check(gdn, inp, normalized, f"bf16 splits={splits}", token_splits=splits)


@pytest.mark.parametrize("normalized", [False, True])
def test_single_frame_and_last_frame_equal_causal(gdn, normalized):
    """The backward history is zero for the last frame: with one frame the
    call is the unidirectional one, and in general the last frame's outputs
    and the terminal states are the unidirectional ones, bit for bit."""
    torch = torch_mod()
    for F in (1, 3):
        inp = make(1, F, 130, normalized, H=2, dtype="bf16", seed=29300 + F)
        t = {k: dev_tensor(inp.get(k)) for k in ("q", "k", "v", "alpha", "beta", "state_in", "z_in")}
        rb = gdn.frame_forward_bidir(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"], t["z_in"],
                                     frame_tokens=130, normalized=normalized)
        if normalized:
            rf = gdn.frame_forward_norm(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"], t["z_in"],
                                        frame_tokens=130)
        else:
            rf = gdn.frame_forward(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"], frame_tokens=130)
        torch.cuda.synchronize()
        last = slice(130 * (F - 1), 130 * F)
        assert torch.equal(rb[0][:, last], rf[0][:, last])
        for x, y in zip(rb[1:], rf[1:]):
            assert torch.equal(x, y)
        if F == 3:
            # the earlier frames do see the later ones
            assert not torch.equal(rb[0][:, :130], rf[0][:, :130])


def test_zero_states_and_no_write(gdn):
    inp = make(0, 3, 70, True, H=2, Dk=64, Dv=64, state="zero", seed=29400)
    check(gdn, inp, True, "norm f32 zero states")
    inp = make(0, 3, 70, False, H=2, Dk=64, Dv=64, state="normal0.02", seed=29401)
    inp["beta"][:] = 0.0
    check(gdn, inp, False, "f32 beta=0 (histories vanish)")


def test_in_place_streaming_bidirectional(gdn):
    """Two calls threading the forward state in place equal the oracle run call
    by call (the backward history spans one call only)."""
    torch = torch_mod()
    inp = make(1, 4, 150, True, H=2, seed=29500)
    N = inp["frame_tokens"]
    state = dev_tensor(inp["state_in"]).clone()
    z = dev_tensor(inp["z_in"]).clone()
    si, zi = inp["state_in"], inp["z_in"]
    for c in range(2):
        sl = slice(2 * N * c, 2 * N * (c + 1))
        part = dict(inp, q=inp["q"][:, sl], k=inp["k"][:, sl], v=inp["v"][:, sl],
                    alpha=inp["alpha"][:, 2 * c:2 * c + 2], beta=inp["beta"][:, sl], state_in=si, z_in=zi)
        t = {key: dev_tensor(part[key]) for key in ("q", "k", "v", "alpha", "beta")}
        out = torch.empty_like(t["v"])
        gdn.frame_forward_bidir(t["q"], t["k"], t["v"], t["alpha"], t["beta"], state, z, frame_tokens=N,
                                normalized=True, out=out, state_out=state, z_out=z)
        ref_o, ref_s, ref_z = oracle_ref(part, True)
        torch.cuda.synchronize()
        eo, es, ez = rel_err(host_f64(out), ref_o), rel_err(host_f64(state), ref_s), rel_err(host_f64(z), ref_z)
        print(f"[bidir parity] streaming call {c}: out {eo:.3e}, state {es:.3e}, z {ez:.3e}", flush=True)
        assert eo < TOL["bf16"] and es < TOL["bf16"] and ez < TOL["bf16"]
        si, zi = ref_s, ref_z


def test_profile_stages_bidir_matches_call(gdn):
    torch = torch_mod()
    inp = make(1, 3, 400, True, H=4, seed=29600)
    t = {k: dev_tensor(inp[k]) for k in ("q", "k", "v", "alpha", "beta", "state_in", "z_in")}
    ws = gdn.frame_workspace(t["q"], t["v"], 400)
    out = torch.empty_like(t["v"])
    st = torch.empty_like(t["state_in"])
    zo = torch.empty_like(t["z_in"])
    ms = gdn.gdn_frame_profile_stages_bidir(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"],
                                            t["z_in"], out, st, zo, ws, 400, normalized=True, reps=3)
    assert len(ms) == 4 and all(x > 0 for x in ms), ms
    o2, s2, z2 = run_gpu(gdn, inp, True, token_splits=0)
    assert torch.equal(out, o2) and torch.equal(st, s2) and torch.equal(zo, z2)


@pytest.mark.parametrize("normalized", [False, True])
def test_three_frame_call_bidirectional_full(gdn, normalized):
    """The paper's streaming call shape (B1 F3 N3520 H16 Dk=Dv=128, bf16), every
    output and the states against the oracle."""
    inp = make(2, 3, 3520, normalized, state="normal0.02", seed=29900 + normalized)
    check(gdn, inp, normalized, f"{'norm ' if normalized else ''}bf16 B1 F3 N3520 H16 D128")


def test_cfg_batch_bidirectional_sampled_heads(gdn):
    inp = make(3, 3, 3520, False, seed=29950)
    check(gdn, inp, False, "bf16 B4 F3 N3520 H20 D64 heads 0,7,19", heads=(0, 7, 19))


@pytest.mark.parametrize("normalized", [False, True])
def test_many_frames_bidirectional(gdn, normalized):
    """40 frames of 16 tokens: the backward sweep and its histories over many
    frames, odd and even sweep lengths in the scan's two-set prefetch."""
    for F in (40, 41):
        inp = make(1, F, 16, normalized, B=1, H=2, dtype="bf16", seed=29980 + F + normalized)
        check(gdn, inp, normalized, f"{'norm ' if normalized else ''}bf16 F{F} N16")
