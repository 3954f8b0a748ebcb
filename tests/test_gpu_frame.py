"""GPU parity of the frame-wise GDN forward (gdn_frame_* through the C ABI)
against the fp64 frame-wise oracle.

Error metric and bounds as for the token-wise path: max|x - x_ref| / max|x_ref|
per tensor, 1e-4 for the fp32 path and 2e-2 for bf16 q/k/v with an fp32
state.  Both sides read the same stored inputs.
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


def run_gpu(gdn, inp, key_scale=None, token_splits=None, state_in="input"):
    t = {k: dev_tensor(inp[k]) for k in ("q", "k", "v", "alpha", "beta")}
    si = dev_tensor(inp["state_in"]) if isinstance(state_in, str) else state_in
    out, st = gdn.frame_forward(t["q"], t["k"], t["v"], t["alpha"], t["beta"], si,
                                frame_tokens=inp["frame_tokens"], key_scale=key_scale,
                                token_splits=token_splits)
    torch_mod().cuda.synchronize()
    return out, st


def oracle_ref(inp, key_scale=None, heads=None):
    sl = slice(None) if heads is None else list(heads)
    si = None if inp["state_in"] is None else inp["state_in"][:, sl]
    return oracle.gdn_frame_forward(inp["q"][:, :, sl], inp["k"][:, :, sl], inp["v"][:, :, sl],
                                    inp["alpha"][:, :, sl], inp["beta"][:, :, sl], si,
                                    frame_tokens=inp["frame_tokens"], key_scale=key_scale)


def check(gdn, inp, label, key_scale=None, token_splits=None, heads=None):
    out, st = run_gpu(gdn, inp, key_scale, token_splits)
    o, s = host_f64(out), host_f64(st)
    ref_o, ref_s = oracle_ref(inp, key_scale, heads)
    if heads is not None:
        o, s = o[:, :, list(heads)], s[:, list(heads)]
    eo, es = rel_err(o, ref_o), rel_err(s, ref_s)
    tol = TOL[inp["dtype"]]
    print(f"[frame parity] {label}: out err {eo:.3e}, state err {es:.3e} (tol {tol:g})", flush=True)
    assert np.isfinite(o).all() and np.isfinite(s).all()
    assert eo < tol, (label, eo)
    assert es < tol, (label, es)
    return out, st


# ---- small shapes: several frames, ragged frames, every (Dk, Dv) pair, both dtypes ----
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("Dk,Dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
@pytest.mark.parametrize("F,N", [(1, 1), (3, 1), (2, 63), (3, 64), (2, 65), (4, 200), (1, 457)])
def test_small_frames(gdn, dtype, Dk, Dv, F, N):
    inp = gdn_inputs.make_frame_inputs(1, F, frame_tokens=N, B=2, H=3, Dk=Dk, Dv=Dv, dtype=dtype,
                                       seed=9100 + F * 1000 + N + Dk + 2 * Dv)
    check(gdn, inp, f"{dtype} Dk{Dk} Dv{Dv} F{F} N{N}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("splits", [1, 2, 3, 5, 100])
def test_token_splits(gdn, dtype, splits):
    """Every split count gives the oracle's result (the summaries are sums over
    disjoint token ranges); the count is capped at one 64-token block per split."""
    inp = gdn_inputs.make_frame_inputs(1, 3, frame_tokens=300, H=2, dtype=dtype, seed=9200 + splits)
    check(gdn, inp, f"{dtype} splits={splits}", token_splits=splits)


def test_explicit_key_scale_and_zero_state(gdn):
    inp = gdn_inputs.make_frame_inputs(0, 3, frame_tokens=130, H=2, Dk=64, Dv=64, state="zero",
                                       seed=9300)
    check(gdn, inp, "f32 key_scale=0.3", key_scale=0.3)
    check(gdn, inp, "f32 key_scale=1.0", key_scale=1.0)


def test_no_write_only_decays(gdn):
    """beta = 0: every frame only decays the state, H_F = prod(alpha) H_0."""
    inp = gdn_inputs.make_frame_inputs(0, 4, frame_tokens=70, H=2, Dk=64, Dv=64, state="normal0.02",
                                       seed=9400)
    inp["beta"][:] = 0.0
    out, st = run_gpu(gdn, inp)
    decay = np.prod(inp["alpha"].astype(np.float64), axis=1)          # [B, H]
    expect = decay[:, :, None, None] * inp["state_in"].astype(np.float64)
    assert rel_err(host_f64(st), expect) < 1e-5
    check(gdn, inp, "f32 beta=0")


def test_zero_decay_resets(gdn):
    """alpha = 0 in frame 1 forgets everything before it: the result from frame 1
    on does not depend on frame 0 or the initial state."""
    inp = gdn_inputs.make_frame_inputs(0, 3, frame_tokens=80, H=2, Dk=64, Dv=64, state="normal0.02",
                                       seed=9500)
    inp["alpha"][:, 1, :] = 0.0
    out_a, st_a = run_gpu(gdn, inp)
    inp2 = dict(inp)
    for key in ("q", "k", "v"):
        x = inp[key].copy()
        x[:, :80] = np.random.default_rng(1).standard_normal(x[:, :80].shape).astype(x.dtype)
        inp2[key] = x
    inp2["state_in"] = 3.0 * inp["state_in"]
    out_b, st_b = run_gpu(gdn, inp2)
    oa, ob = host_f64(out_a)[:, 80:], host_f64(out_b)[:, 80:]
    assert rel_err(ob, oa) < 1e-5 and rel_err(host_f64(st_b), host_f64(st_a)) < 1e-5
    check(gdn, inp, "f32 alpha_1=0")


def test_in_place_state_and_streaming(gdn):
    """Two calls threading the state in place (state_in == state_out) equal one
    call over all frames, within the tolerance of either against the oracle."""
    torch = torch_mod()
    inp = gdn_inputs.make_frame_inputs(1, 4, frame_tokens=150, H=2, seed=9600)
    N = inp["frame_tokens"]
    ref_o, ref_s = oracle_ref(inp)
    state = dev_tensor(inp["state_in"]).clone()
    outs = []
    for c in range(2):
        sl = slice(2 * N * c, 2 * N * (c + 1))
        part = dict(inp, q=inp["q"][:, sl], k=inp["k"][:, sl], v=inp["v"][:, sl],
                    alpha=inp["alpha"][:, 2 * c:2 * c + 2], beta=inp["beta"][:, sl])
        t = {k: dev_tensor(part[k]) for k in ("q", "k", "v", "alpha", "beta")}
        out, st = torch_mod().empty_like(t["v"]), state
        gdn.frame_forward(t["q"], t["k"], t["v"], t["alpha"], t["beta"], state, frame_tokens=N,
                          out=out, state_out=state)
        outs.append(out)
    torch.cuda.synchronize()
    o = np.concatenate([host_f64(x) for x in outs], axis=1)
    eo, es = rel_err(o, ref_o), rel_err(host_f64(state), ref_s)
    print(f"[frame parity] streaming in place: out {eo:.3e}, state {es:.3e}", flush=True)
    assert eo < TOL["bf16"] and es < TOL["bf16"]


def test_deterministic(gdn):
    inp = gdn_inputs.make_frame_inputs(1, 3, frame_tokens=500, H=4, seed=9700)
    o1, s1 = run_gpu(gdn, inp)
    o2, s2 = run_gpu(gdn, inp)
    torch = torch_mod()
    assert torch.equal(o1, o2) and torch.equal(s1, s2)


def test_profile_stages_matches_call(gdn):
    torch = torch_mod()
    inp = gdn_inputs.make_frame_inputs(1, 3, frame_tokens=400, H=4, seed=9800)
    t = {k: dev_tensor(inp[k]) for k in ("q", "k", "v", "alpha", "beta", "state_in")}
    ws = gdn.frame_workspace(t["q"], t["v"], 400)
    out = torch.empty_like(t["v"])
    st = torch.empty_like(t["state_in"])
    ms = gdn.gdn_frame_profile_stages(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"],
                                      out, st, ws, 400, reps=3)
    assert len(ms) == 4 and all(x > 0 for x in ms), ms
    o2, s2 = run_gpu(gdn, inp, token_splits=0)
    assert torch.equal(out, o2) and torch.equal(st, s2)


# ---- the paper's streaming call: 3 latent frames of 44 x 80 tokens, 16 heads, D = 128 ----
def test_three_frame_call_full(gdn):
    """B=1, F=3, N=3520, H=16, Dk=Dv=128, bf16: every output and the whole
    state against the oracle, in the launch configuration the benchmark uses."""
    inp = gdn_inputs.make_frame_inputs(2, 3, seed=9900)
    check(gdn, inp, "bf16 B1 F3 N3520 H16 D128")


def test_cfg_batch_frames_sampled_heads(gdn):
    """B=4, H=20, Dk=Dv=64, 3 frames of 3520 tokens with fast-forgetting decays;
    the oracle on a sample of heads."""
    inp = gdn_inputs.make_frame_inputs(3, 3, seed=9950)
    check(gdn, inp, "bf16 B4 F3 N3520 H20 D64 heads 0,7,19", heads=(0, 7, 19))


def test_rejects_bad_frames(gdn):
    torch = torch_mod()
    q = torch.zeros(1, 100, 2, 64, device="cuda")
    with pytest.raises(ValueError):
        gdn.frame_forward(q, q, q, torch.zeros(1, 3, 2, device="cuda"), torch.zeros(1, 100, 2, device="cuda"),
                          frame_tokens=33)
    with pytest.raises(ValueError):
        gdn.frame_forward(q, q, q, torch.zeros(1, 100, 2, device="cuda"), torch.zeros(1, 100, 2, device="cuda"),
                          frame_tokens=50)
