"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, sizes workspaces, and rejects bad arguments before touching
the GPU (no compute call is made here)."""
import ctypes
import os
import re

import pytest

import paper_2605_30409_amd as gdn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gdn.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_]+\s*\**\s*(gdn_[a-z0-9_]+)\s*\(", src, flags=re.M)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) == 7 and "gdn_workspace_bytes" in names, names
    lib = ctypes.CDLL(gdn.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    assert gdn.gdn_status_string(0) == "ok"
    for s in range(-7, 0):
        assert gdn.gdn_status_string(s) not in ("ok", "unknown status")
    assert gdn.gdn_status_string(-99) == "unknown status"


def test_workspace_bytes():
    n = gdn.gdn_workspace_bytes(1, 16, 3520, 128, 128, 64, True)
    nch = 16 * 55
    # g + W + Kt + Ut + Hs + Us (each region 256-byte aligned)
    expect = nch * 64 * 8 + nch * 2 * (64 * 128 * 4 + 128 * 128)
    assert expect <= n < expect + 6 * 256
    assert gdn.gdn_workspace_bytes(1, 16, 3520, 128, 128, 64, False) > n
    assert gdn.gdn_workspace_bytes(1, 16, 3520, 96, 128, 64, True) == 0
    assert gdn.gdn_workspace_bytes(1, 16, 3520, 128, 128, 32, True) == 0
    assert gdn.gdn_workspace_bytes(0, 16, 3520, 128, 128, 64, True) == 0
    assert gdn.gdn_workspace_bytes(1, 16, 0, 128, 128, 64, True) == 0
    # ragged T rounds up to whole chunks
    assert gdn.gdn_workspace_bytes(1, 2, 65, 64, 64, 64, True) == gdn.gdn_workspace_bytes(1, 2, 128, 64, 64, 64, True)


# Fake, never-dereferenced device addresses: validation fails before any HIP call.
BASE = 1 << 40
MB = 1 << 20


def call(fn, q=BASE, k=BASE + 64 * MB, v=BASE + 128 * MB, a=BASE + 192 * MB, b=BASE + 200 * MB,
         si=None, o=BASE + 256 * MB, so=None, B=1, H=2, T=256, Dk=64, Dv=64, chunk=64, ws=None,
         ws_bytes=0):
    L = gdn.lib()
    args = [q, k, v, a, b, si, o, so, B, H, T, Dk, Dv, chunk]
    if fn.endswith("_ws"):
        args += [ws, ws_bytes]
    return getattr(L, fn)(*args, None)


@pytest.mark.parametrize("fn", ["gdn_chunk_forward", "gdn_chunk_forward_f32",
                                "gdn_chunk_forward_ws", "gdn_chunk_forward_f32_ws"])
def test_validation_errors(fn):
    assert call(fn, q=None) == -1
    assert call(fn, o=None) == -1
    assert call(fn, a=None) == -1
    assert call(fn, T=0) == -2
    assert call(fn, B=0) == -2
    assert call(fn, H=300, B=300) == -2
    assert call(fn, Dk=96) == -3
    assert call(fn, Dv=32) == -3
    assert call(fn, chunk=128) == -3
    assert call(fn, k=BASE + 64 * MB + 8) == -6
    assert call(fn, o=BASE + 4096) == -7                 # out overlaps q
    assert call(fn, so=BASE + 64 * MB) == -7             # state_out overlaps k
    assert call(fn, si=BASE + 300 * MB, so=BASE + 300 * MB + 4096) == -7  # partial state overlap
    if fn.endswith("_ws"):
        assert call(fn) == -4                            # no workspace
        assert call(fn, ws=BASE + 512 * MB, ws_bytes=100) == -4
        assert call(fn, ws=BASE + 512 * MB + 16, ws_bytes=1 << 30) == -4   # misaligned


def test_binding_rejects_bad_tensors_on_cpu():
    import torch
    q = torch.zeros(1, 64, 2, 64)
    with pytest.raises(ValueError):
        gdn.forward(q, q, q, torch.zeros(1, 64, 2), torch.zeros(1, 64, 2))
    with pytest.raises(TypeError):
        gdn.forward(q.half(), q, q, torch.zeros(1, 64, 2), torch.zeros(1, 64, 2))
