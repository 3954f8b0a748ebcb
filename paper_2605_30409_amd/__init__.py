"""MI355X (gfx950) gated delta-rule forward: HIP kernels behind a C ABI.

The compute lives in ``libgdn.so`` (``csrc/``), declared in ``include/gdn.h``;
:mod:`.gdn` is the thin ctypes binding with the same entry-point names.  The
operations: the token-wise chunk forward (``forward``, ``gdn_chunk_forward*``),
the frame-wise forward (``frame_forward``, ``gdn_frame_forward*``), the
frame-wise forward with the normalizer (``frame_forward_norm``), the
bidirectional frame-wise forward (``frame_forward_bidir``) and the fused
operator with its prologue and epilogue (``frame_forward_fused``).
"""
from .gdn import (CHUNK, FRAME_STAGE_NAMES, STAGE_NAMES, GdnError, LIB_PATH,  # noqa: F401
                  default_key_scale, forward, frame_forward, frame_forward_bidir, frame_forward_fused,
                  frame_forward_norm, frame_workspace, fused_workspace, gdn_chunk_forward, gdn_frame_profile_stages_bidir,
                  gdn_frame_profile_stages_fused,
                  gdn_frame_profile_stages_norm,
                  gdn_chunk_forward_ex, gdn_chunk_forward_f32, gdn_chunk_forward_f32_ws,
                  gdn_chunk_forward_ws, gdn_chunk_forward_noalloc, gdn_frame_forward_ex, gdn_frame_profile_stages,
                  gdn_frame_token_splits, gdn_frame_workspace_bytes, gdn_profile_stages,
                  gdn_scan_group_size, gdn_status_string, gdn_workspace_bytes,
                  gdn_workspace_bytes_ex, lib, workspace)
