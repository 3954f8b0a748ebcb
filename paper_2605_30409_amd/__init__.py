"""MI355X (gfx950) gated delta-rule chunk forward: HIP kernels behind a C ABI.

The compute lives in ``libgdn.so`` (``csrc/``), declared in ``include/gdn.h``;
:mod:`.gdn` is the thin ctypes binding with the same entry-point names.
"""
from .gdn import (CHUNK, STAGE_NAMES, GdnError, LIB_PATH, forward, gdn_chunk_forward,  # noqa: F401
                  gdn_chunk_forward_ex, gdn_chunk_forward_f32, gdn_chunk_forward_f32_ws,
                  gdn_chunk_forward_ws, gdn_profile_stages, gdn_scan_group_size, gdn_status_string,
                  gdn_workspace_bytes, gdn_workspace_bytes_ex, lib, workspace)
