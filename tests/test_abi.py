"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, sizes workspaces, and rejects bad arguments before touching
the GPU (no compute call is made here)."""
import ctypes
import os
import re
import sys

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
    assert len(names) == 31 and "gdn_workspace_bytes" in names and "gdn_frame_forward" in names, names
    lib = ctypes.CDLL(gdn.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    assert gdn.gdn_status_string(0) == "ok"
    for s in range(-7, 0):
        assert gdn.gdn_status_string(s) not in ("ok", "unknown status")
    assert gdn.gdn_status_string(-99) == "unknown status"


def test_scan_group_size():
    sg = gdn.gdn_scan_group_size
    f32 = dict(is_bf16=False)
    # bf16: one group once the streams give >= 64 column tiles, or up to 64 chunks
    assert sg(1, 16, 3520, 128, 128) == 55               # 55 chunks
    assert sg(1, 16, 10560, 128, 128) == 165             # 16 streams x 8 column tiles
    assert sg(1, 32, 42240, 128, 128) == 660
    assert sg(4, 20, 10560, 64, 64) == 165               # 80 streams x 4 column tiles
    assert sg(1, 4, 10560, 128, 128) == 13               # 32 column tiles: ~sqrt(165)
    assert sg(1, 2, 4097, 64, 64) == 8                   # 65 chunks, 8 column tiles
    # fp32: one group up to 64 chunks or when the streams fill the chip (512 tiles)
    assert sg(1, 16, 3520, 128, 128, **f32) == 55
    assert sg(1, 16, 4097, 128, 128, **f32) == 8         # 65 chunks: round(sqrt(65))
    assert sg(1, 16, 10560, 128, 128, **f32) == 13       # 165 chunks
    assert sg(1, 32, 42240, 128, 128, **f32) == 26       # 660 chunks
    assert sg(4, 20, 10560, 64, 64, **f32) == 13         # 80 streams x 4 column tiles
    assert sg(8, 16, 10560, 128, 128, **f32) == 165      # 128 streams x 8 column tiles fill the chip
    assert sg(1, 2, 1, 64, 64) == 1
    assert sg(1, 16, 3520, 128, 128, scan_group=7) == 7
    assert sg(1, 16, 3520, 128, 128, scan_group=1000) == 55
    assert sg(1, 16, 10560, 128, 128, scan_group=-3) == 165
    assert sg(1, 16, 10560, 128, 128, scan_group=-3, **f32) == 13
    assert sg(1, 16, 0, 128, 128) == 0
    assert sg(1, 16, 64, 128, 128, chunk=32) == 0
    assert sg(1, 16, 64, 96, 128) == 0


def test_workspace_bytes():
    nch = 16 * 55
    # g, gate records (key decay factors and g_C), -W, Ut, Hs, Us
    gates = nch * 64 * 8 + nch * 68 * 4
    base = gates + nch * 2 * (64 * 128 * 2 + 128 * 128 + 128 * 64)
    # one scan group on the bf16 path: the output is fused into the scan and the
    # last two regions hold the scaled queries (64 x 128) and scores (64 x 64)
    fused = gates + nch * 2 * (64 * 128 * 3 + 64 * 64)
    n = gdn.gdn_workspace_bytes(1, 16, 3520, 128, 128, 64, True)
    assert fused <= n < fused + 10 * 256
    assert n == gdn.gdn_workspace_bytes_ex(1, 16, 3520, 128, 128, 64, True, 0)
    n32 = gdn.gdn_workspace_bytes(1, 16, 3520, 128, 128, 64, False)   # fp32: per-chunk states
    base32 = gates + nch * 4 * (64 * 128 * 2 + 128 * 128 + 128 * 64)
    assert base32 <= n32 < base32 + 10 * 256
    # 11 groups of 5 chunks add N (bf16), Psi^T, log Gamma and entry states (fp32)
    ngr = 16 * 11
    grouped = gdn.gdn_workspace_bytes_ex(1, 16, 3520, 128, 128, 64, True, 5)
    expect = base + ngr * (128 * 128 * 2 + 128 * 128 * 4 * 2 + 8)
    assert expect <= grouped < expect + 10 * 256
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
    if fn.endswith("_ex"):
        args += [1, 0]                                   # bf16, library group size
    if fn.endswith("_ws") or fn.endswith("_ex"):
        args += [ws, ws_bytes]
    return getattr(L, fn)(*args, None)


@pytest.mark.parametrize("fn", ["gdn_chunk_forward", "gdn_chunk_forward_f32",
                                "gdn_chunk_forward_ws", "gdn_chunk_forward_f32_ws",
                                "gdn_chunk_forward_ex", "gdn_chunk_forward_noalloc"])
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
    if fn.endswith("_ws") or fn.endswith("_ex"):
        assert call(fn) == -4                            # no workspace
        assert call(fn, ws=BASE + 512 * MB, ws_bytes=100) == -4
        assert call(fn, ws=BASE + 512 * MB + 16, ws_bytes=1 << 30) == -4   # misaligned


@pytest.mark.parametrize("is_bf16", [1, 0])
@pytest.mark.parametrize("Dk,Dv", [(64, 64), (128, 128), (64, 128), (128, 64)])
def test_workspace_regions_cover_kernel_indexing(is_bf16, Dk, Dv):
    """Every workspace region spans what the kernels index in it, for every
    path: one scan group (fused output on bf16), grouped scans with short last
    groups, ragged T, batches, many heads."""
    L = gdn.lib()
    for B, H in ((1, 1), (1, 16), (2, 3), (4, 20), (1, 32), (8, 16)):
        for T in (1, 63, 64, 65, 200, 1500, 3520, 3557, 10560, 42240):
            nc = -(-T // 64)
            for g in sorted({0, 1, 2, 7, 13, nc, nc + 5}):
                rc = L.gdn_workspace_check(B, H, T, Dk, Dv, 64, is_bf16, g)
                assert rc == 0, (B, H, T, Dk, Dv, is_bf16, g, rc)
    assert L.gdn_workspace_check(1, 1, 0, 64, 64, 64, 1, 0) == -2
    assert L.gdn_workspace_check(1, 1, 64, 96, 64, 64, 1, 0) == -3


def test_noalloc_rejects_workspace_beyond_its_array():
    """The allocation-free call returns GDN_ERR_WORKSPACE, before any HIP call,
    when the shape's workspace exceeds its static array (64 MiB): one 1280x704
    frame at H = 16 fits, twelve frames at H = 32 do not."""
    limit = 64 << 20
    assert gdn.gdn_workspace_bytes(1, 16, 3520, 128, 128, 64, True) <= limit
    big = dict(B=1, H=32, T=42240, Dk=128, Dv=128)
    assert gdn.gdn_workspace_bytes(1, 32, 42240, 128, 128, 64, True) > limit
    n = big["B"] * big["T"] * big["H"] * 128 * 2
    assert call("gdn_chunk_forward_noalloc", q=BASE, k=BASE + n, v=BASE + 2 * n, a=BASE + 3 * n,
                b=BASE + 3 * n + (1 << 30), o=BASE + 4 * n, **big) == -4


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """No fallback: without the built library every entry point raises."""
    from paper_2605_30409_amd import gdn as binding
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", str(tmp_path / "libgdn.so"))
    with pytest.raises(ImportError):
        binding.lib()
    with pytest.raises(ImportError):
        binding.gdn_status_string(0)
    with pytest.raises(ImportError):
        binding.gdn_workspace_bytes(1, 2, 64, 64, 64)


def test_binding_rejects_bad_tensors_on_cpu():
    import torch
    q = torch.zeros(1, 64, 2, 64)
    with pytest.raises(ValueError):
        gdn.forward(q, q, q, torch.zeros(1, 64, 2), torch.zeros(1, 64, 2))
    with pytest.raises(TypeError):
        gdn.forward(q.half(), q, q, torch.zeros(1, 64, 2), torch.zeros(1, 64, 2))


def test_frame_token_splits_and_workspace():
    ts = gdn.gdn_frame_token_splits
    # library choice: summary workgroups (one per split) within 256
    assert ts(1, 16, 3, 3520, 128, 128) == 5             # 48 (frame, head) units
    assert ts(1, 16, 1, 3520, 128, 128) == 14            # 16 units: 16 splits of 4 blocks -> 14
    assert ts(4, 20, 3, 3520, 64, 64) == 1               # 240 units
    assert ts(1, 2, 1, 3520, 64, 64) == 55               # capped at one 64-token block per split
    assert ts(1, 16, 3, 3520, 128, 128, 2) == 2
    assert ts(1, 16, 3, 3520, 128, 128, 1000) == 55
    assert ts(1, 16, 3, 3520, 128, 128, 13) == 11        # 5 blocks per split, none empty
    assert ts(1, 2, 1, 100, 64, 64, 5) == 2
    assert ts(1, 2, 1, 1, 64, 64) == 1
    assert ts(0, 2, 1, 1, 64, 64) == 0
    assert ts(1, 2, 1, 1, 96, 64) == 0
    wb = gdn.gdn_frame_workspace_bytes
    bhf = 16 * 3
    n = wb(1, 16, 3, 3520, 128, 128, True, 1)           # one split: no partial sums
    # G fragments (bf16), A tiles (fp32), state fragments (bf16) and backward
    # histories (fp32), the last three with room for the normalizer's extra
    # 16-column tile
    expect = bhf * (128 * 128 * 2 + 128 * 144 * (4 + 2 + 4) + 128 * 128 * 2)   # + unrotated-key G (fused)
    assert expect <= n < expect + 8 * 256
    assert wb(1, 16, 3, 3520, 128, 128, True, 2) - n >= bhf * 2 * 128 * (2 * 128 + 144) * 4
    assert wb(1, 16, 3, 3520, 128, 128, False, 1) > n
    assert wb(1, 16, 3, 0, 128, 128, True, 0) == 0
    assert wb(1, 16, 3, 3520, 128, 32, True, 0) == 0
    # the fused operator: bf16 as above; fp32 also keeps q~, q^, k~, k^ and the
    # gated readout for every token row
    fb = gdn.lib().gdn_frame_fused_workspace_bytes
    assert fb(1, 16, 3, 3520, 128, 128, 1, 1) == n
    base32 = wb(1, 16, 3, 3520, 128, 128, False, 1)
    rows = 16 * 3 * 3520
    assert base32 + rows * (4 * 128 + 128) * 4 <= fb(1, 16, 3, 3520, 128, 128, 0, 1) < \
        base32 + rows * (4 * 128 + 128) * 4 + 5 * 256
    assert fb(1, 16, 3, 3520, 96, 128, 0, 1) == 0


def fcall(fn, q=BASE, k=BASE + 64 * MB, v=BASE + 128 * MB, a=BASE + 192 * MB, b=BASE + 200 * MB,
          si=None, o=BASE + 256 * MB, so=None, B=1, H=2, F=2, N=100, Dk=64, Dv=64, ks=0.1,
          ws=None, ws_bytes=0):
    L = gdn.lib()
    args = [q, k, v, a, b, si, o, so, B, H, F, N, Dk, Dv, ctypes.c_float(ks)]
    if fn.endswith("_ex"):
        args += [1, 0, ws, ws_bytes]
    return getattr(L, fn)(*args, None)


@pytest.mark.parametrize("fn", ["gdn_frame_forward", "gdn_frame_forward_f32", "gdn_frame_forward_ex"])
def test_frame_validation_errors(fn):
    assert fcall(fn, q=None) == -1
    assert fcall(fn, a=None) == -1
    assert fcall(fn, o=None) == -1
    assert fcall(fn, F=0) == -2
    assert fcall(fn, N=0) == -2
    assert fcall(fn, H=300, B=300) == -2
    assert fcall(fn, F=1 << 16, N=1 << 16) == -2         # token index beyond int
    assert fcall(fn, Dk=96) == -3
    assert fcall(fn, Dv=32) == -3
    assert fcall(fn, b=BASE + 200 * MB + 4) == -6
    assert fcall(fn, o=BASE + 4096) == -7                # out overlaps q
    assert fcall(fn, o=BASE + 192 * MB) == -7            # out overlaps alpha
    assert fcall(fn, so=BASE + 128 * MB) == -7           # state_out overlaps v
    assert fcall(fn, si=BASE + 300 * MB, so=BASE + 300 * MB + 4096) == -7
    if fn.endswith("_ex"):
        assert fcall(fn) == -4
        assert fcall(fn, ws=BASE + 512 * MB, ws_bytes=100) == -4
        assert fcall(fn, ws=BASE + 512 * MB + 16, ws_bytes=1 << 30) == -4


def test_frame_binding_rejects_bad_tensors_on_cpu():
    import torch
    q = torch.zeros(1, 100, 2, 64)
    with pytest.raises(ValueError):
        gdn.frame_forward(q, q, q, torch.zeros(1, 2, 2), torch.zeros(1, 100, 2), frame_tokens=50)


def ncall(fn, q=BASE, k=BASE + 64 * MB, v=BASE + 128 * MB, a=BASE + 192 * MB, b=BASE + 200 * MB,
          si=None, zi=None, o=BASE + 256 * MB, so=None, zo=None, B=1, H=2, F=2, N=100, Dk=64, Dv=64,
          ws=None, ws_bytes=0):
    L = gdn.lib()
    args = [q, k, v, a, b, si, zi, o, so, zo, B, H, F, N, Dk, Dv, ctypes.c_float(0.1),
            ctypes.c_float(1e-6), 1]
    if "_bidir" in fn:
        args += [1]                                      # normalized
    if fn.endswith("_ex"):
        args += [0, ws, ws_bytes]
    return getattr(L, fn)(*args, None)


@pytest.mark.parametrize("fn", ["gdn_frame_forward_norm", "gdn_frame_forward_norm_ex",
                                "gdn_frame_forward_bidir", "gdn_frame_forward_bidir_ex"])
def test_frame_norm_validation_errors(fn):
    Z = BASE + 320 * MB
    assert ncall(fn, q=None) == -1
    assert ncall(fn, F=0) == -2
    assert ncall(fn, Dk=96) == -3
    assert ncall(fn, zi=Z + 4) == -6
    assert ncall(fn, zo=BASE + 64 * MB) == -7            # z_out overlaps k
    assert ncall(fn, zo=BASE + 256 * MB + 64) == -7      # z_out overlaps out
    assert ncall(fn, zi=Z, zo=Z + 16) == -7              # partial overlap of z_in and z_out
    assert ncall(fn, zi=BASE + 256 * MB) == -7           # out overlaps z_in
    assert ncall(fn, si=Z, zo=Z) == -7                   # z_out overlaps state_in
    assert ncall(fn, so=Z, zo=Z + 1024) == -7            # z_out overlaps state_out
    if fn.endswith("_ex"):
        assert ncall(fn, zi=Z, zo=Z) == -4               # in place is fine; no workspace
        assert ncall(fn, ws=BASE + 512 * MB, ws_bytes=100) == -4


def test_frame_norm_binding_rejects_bad_z_on_cpu():
    import torch
    q = torch.zeros(1, 100, 2, 64)
    with pytest.raises(ValueError):
        gdn.frame_forward_norm(q, q, q, torch.zeros(1, 2, 2), torch.zeros(1, 100, 2),
                               z_in=torch.zeros(1, 2, 32), frame_tokens=50)


@pytest.mark.parametrize("fn", ["gdn_frame_forward_bidir", "gdn_frame_forward_bidir_ex"])
def test_frame_bidir_unnormalized_ignores_z(fn):
    """normalized == 0: z pointers are not validated (they are not used)."""
    L = gdn.lib()
    args = [BASE, BASE + 64 * MB, BASE + 128 * MB, BASE + 192 * MB, BASE + 200 * MB, None,
            BASE + 4, BASE + 256 * MB, None, BASE + 64 * MB, 1, 2, 2, 100, 64, 64, ctypes.c_float(0.1),
            ctypes.c_float(1e-6), 1, 0]
    if fn.endswith("_ex"):
        args += [0, None, 0]
        assert getattr(L, fn)(*args, None) == -4         # reaches the workspace check
    else:
        args[7] = BASE + 4096                             # out overlaps q: rejected before any launch
        assert getattr(L, fn)(*args, None) == -7


def test_frame_bidir_profile_rejects_in_place():
    L = gdn.lib()
    ms = (ctypes.c_float * 4)()
    S = BASE + 300 * MB
    args = [BASE, BASE + 64 * MB, BASE + 128 * MB, BASE + 192 * MB, BASE + 200 * MB, S, None,
            BASE + 256 * MB, S, None, 1, 2, 2, 100, 64, 64, ctypes.c_float(0.1), ctypes.c_float(1e-6), 1, 0,
            0, None, 0, 3, ms]
    assert L.gdn_frame_profile_stages_bidir(*args, None) == -7


def ucall(fn, q=BASE, k=BASE + 64 * MB, v=BASE + 128 * MB, g=BASE + 160 * MB, w=BASE + 176 * MB,
          a=BASE + 192 * MB, b=BASE + 200 * MB, gq=BASE + 208 * MB, gk=BASE + 209 * MB, fr=BASE + 210 * MB,
          ax=BASE + 211 * MB, si=None, zi=None, o=BASE + 256 * MB, so=None, zo=None, B=1, H=2, F=2, N=100,
          Dk=64, Dv=64, lat_w=10, ws=None, ws_bytes=0):
    L = gdn.lib()
    args = [q, k, v, g, w, a, b, gq, gk, fr, ax, si, zi, o, so, zo, B, H, F, N, Dk, Dv, lat_w, 0,
            ctypes.c_float(0.1), ctypes.c_float(1e-6), ctypes.c_float(1e-6), 0]
    if fn.endswith("_ex"):
        args += [0, ws, ws_bytes]
    return getattr(L, fn)(*args, None)


@pytest.mark.parametrize("fn", ["gdn_frame_forward_fused", "gdn_frame_forward_fused_ex",
                                "gdn_frame_forward_fused_f32", "gdn_frame_forward_fused_f32_ex"])
def test_frame_fused_validation_errors(fn):
    assert ucall(fn, g=None) == -1
    assert ucall(fn, w=None) == -1
    assert ucall(fn, ax=None) == -1
    assert ucall(fn, lat_w=0) == -2
    assert ucall(fn, Dk=96) == -3
    assert ucall(fn, g=BASE + 160 * MB + 8) == -6
    assert ucall(fn, o=BASE + 176 * MB) == -7            # out overlaps w_o
    assert ucall(fn, so=BASE + 208 * MB) == -7           # state_out overlaps gain_q
    if fn.endswith("_ex"):
        assert ucall(fn) == -4


def test_frame_fused_binding_rejects_mixed_types_and_host_tensors():
    import torch
    q = torch.zeros(1, 100, 2, 64)
    args = (torch.zeros(1, 2, 2), torch.zeros(1, 100, 2), torch.ones(2, 64), torch.ones(2, 64), torch.ones(32),
            torch.zeros(32, dtype=torch.int32))
    with pytest.raises(ValueError):       # host tensors
        gdn.frame_forward_fused(q, q, q, q, torch.zeros(2, 64, 64), *args, frame_tokens=50, lat_w=10)
    qb = q.to(torch.bfloat16)
    with pytest.raises(ValueError):       # bf16 q with an fp32 gate
        gdn.frame_forward_fused(qb, qb, qb, q, torch.zeros(2, 64, 64, dtype=torch.bfloat16), *args,
                                frame_tokens=50, lat_w=10)


_FAILED_LAUNCH = r"""
import sys
sys.path.insert(0, {root!r})
import paper_2605_30409_amd as gdn
L = gdn.lib()
BASE, MB = 1 << 40, 1 << 20
n = gdn.gdn_workspace_bytes(1, 2, 130, 64, 64)
args = (BASE, BASE + 64 * MB, BASE + 128 * MB, BASE + 192 * MB, BASE + 200 * MB, None, BASE + 256 * MB, None,
        1, 2, 130, 64, 64, 64)
print(L.gdn_chunk_forward_ws(*args, BASE + 512 * MB, n, None), L.gdn_chunk_forward(*args, None))
"""


def test_failed_launch_returns_hip_error():
    """Arguments that pass validation on a host whose HIP launches fail (no GPU):
    both the explicit-workspace and the cached-workspace calls return
    GDN_ERR_HIP (-5) instead of crashing or reporting success.  Runs in a child
    process (the HIP runtime keeps its failed state), and only where no GPU is
    visible: there the fake addresses are never dereferenced."""
    import subprocess
    from conftest import gpu_available
    if gpu_available():
        pytest.skip("a GPU is visible: the fake addresses would be launched on")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", _FAILED_LAUNCH.format(root=root)], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.split() == ["-5", "-5"]  # GDN_ERR_HIP
