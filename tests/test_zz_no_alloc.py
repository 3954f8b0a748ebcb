"""GPU: the allocation-free entry point (static device workspace) against the
explicit-workspace call, through the C ABI: bitwise equal outputs and states,
on two calls in a row, the second on a smaller input (the array keeps the first
call's contents)."""
import numpy as np
import pytest

import gdn_inputs

pytestmark = pytest.mark.gpu


def dev(a):
    import torch
    if a is None:
        return None
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("shapes", [((1, 3520, 16, 128, 128), (2, 333, 3, 64, 128)),
                                    ((1, 1000, 4, 128, 64), (1, 65, 2, 64, 64))])
def test_noalloc_matches_explicit_workspace(gdn, shapes):
    import torch
    for i, (B, T, H, Dk, Dv) in enumerate(shapes):
        inp = gdn_inputs.make_inputs(1, B=B, T=T, H=H, Dk=Dk, Dv=Dv, seed=4200 + 17 * i + T)
        t = {k: dev(inp[k]) for k in ("q", "k", "v", "alpha", "beta", "state_in")}
        out_ref = torch.empty((B, T, H, Dv), dtype=torch.bfloat16, device="cuda")
        st_ref = torch.empty((B, H, Dk, Dv), dtype=torch.float32, device="cuda")
        ws = gdn.workspace(t["q"], t["v"])
        gdn.gdn_chunk_forward_ws(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"], out_ref, st_ref, ws)
        out = torch.full_like(out_ref, float("nan"))
        st = torch.full_like(st_ref, float("nan"))
        gdn.gdn_chunk_forward_noalloc(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"], out, st)
        torch.cuda.synchronize()
        print(f"[noalloc] call {i}: B{B} T{T} H{H} Dk{Dk} Dv{Dv}", flush=True)
        assert torch.equal(out, out_ref), f"call {i}: out differs"
        assert torch.equal(st, st_ref), f"call {i}: state differs"
