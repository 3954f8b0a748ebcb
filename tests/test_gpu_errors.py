"""GPU: a HIP error the caller left pending is not reported as the GDN call's.

The library reports GDN_ERR_HIP only for errors its own launches return
(hipLaunchKernel's status); it neither reads nor clears the thread's pending
HIP error."""
import ctypes

import numpy as np
import pytest

import gdn_inputs

pytestmark = pytest.mark.gpu


def test_pending_error_not_attributed(gdn):
    import torch
    inp = gdn_inputs.make_inputs(1, T=130, H=2)
    t = {k: torch.from_numpy(np.ascontiguousarray(inp[k]).view(np.int16)).view(torch.bfloat16).cuda()
         if inp[k].dtype == np.uint16 else torch.from_numpy(inp[k]).cuda()
         for k in ("q", "k", "v", "alpha", "beta", "state_in")}
    B, T, H, Dk = t["q"].shape
    Dv = t["v"].shape[-1]
    out_ref, st_ref = gdn.forward(t["q"], t["k"], t["v"], t["alpha"], t["beta"], t["state_in"])
    out = torch.empty_like(out_ref)
    st = torch.empty_like(st_ref)
    ws = gdn.workspace(t["q"], t["v"])
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    hip = ctypes.CDLL("libamdhip64.so.7")   # the runtime already loaded in this process
    hip.hipSetDevice.argtypes = [ctypes.c_int]
    hip.hipGetLastError()
    p = lambda x: ctypes.c_void_p(x.data_ptr())
    # leave an invalid-device error pending, then call straight through the C ABI
    assert hip.hipSetDevice(10 ** 6) != 0
    rc = gdn.lib().gdn_chunk_forward_ws(p(t["q"]), p(t["k"]), p(t["v"]), p(t["alpha"]), p(t["beta"]),
                                        p(t["state_in"]), p(out), p(st), B, H, T, Dk, Dv, 64, p(ws), ws.numel(),
                                        ctypes.c_void_p(stream.cuda_stream))
    hip.hipGetLastError()                   # clear what this test left pending
    torch.cuda.synchronize()
    assert rc == 0, gdn.gdn_status_string(rc)
    assert torch.equal(out, out_ref) and torch.equal(st, st_ref)
