/*
 * gdn.h -- C ABI of the MI355X (gfx950) gated delta-rule chunk forward.
 *
 * Operation (paper: Section "Hybrid Architecture", equation gdn_combined, and
 * Section "Frame-wise Gated DeltaNet", equations appendix_gdn_kv_update /
 * appendix_gdn_kv_compact, applied with one token per update; readout as in
 * equation appendix_gdn_readout without the normalizer, gate or projection):
 *
 *   for each batch b and head h independently, for t = 0 .. T-1:
 *     S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
 *     o_t = S_t q_t
 *
 * S_{-1} is state_in, and the terminal S_{T-1} is written to state_out: only
 * that terminal state is carried from one streaming call to the next
 * (subsection "Streaming cache").  The state is stored transposed, as
 * H = S^T with shape [Dk][Dv] per (b, h), the orientation in which the paper's
 * kernel section writes the scan (S_f = alpha_f P_f S_{f-1} + A_f).
 *
 * The work is evaluated chunk by chunk (chunks of `chunk` tokens): a per-chunk
 * WY/UT transform, a scan of the state across chunks, and a per-chunk output
 * pass.  Long sequences split the scan into groups of consecutive chunks: the
 * transfer map of every group (its product of per-chunk transitions and its
 * zero-start state) is formed in parallel, a short sequential scan over the
 * groups yields each group's entry state, and the chunk states inside all
 * groups then follow in parallel.  This is an exact rewrite of the
 * recurrence; results differ from it only by rounding (and, slightly, with
 * the group size).
 *
 * Layouts (all contiguous, row-major, 64-bit indexed):
 *   q, k      [B][T][H][Dk]      bf16 (gdn_chunk_forward*) or fp32 (*_f32*)
 *   v, out    [B][T][H][Dv]      same element type as q
 *   alpha     [B][T][H]          fp32, decay gate, expected in [0, 1]
 *   beta      [B][T][H]          fp32, write gate, expected in [0, 1] (any finite value works)
 *   state_in  [B][H][Dk][Dv]     fp32, or NULL for a zero initial state
 *   state_out [B][H][Dk][Dv]     fp32, or NULL to drop the terminal state
 *
 * Pointers q .. state_out are DEVICE pointers on the current HIP device,
 * owned by the caller and 16-byte aligned.  state_in == state_out (in-place
 * streaming) is allowed; `out` and `state_out` must not overlap any input
 * otherwise.  Supported shapes: B, H, T >= 1; Dk, Dv in {64, 128};
 * chunk == 64.  T need not be a multiple of the chunk: the tail is processed
 * as if padded with alpha = 1, beta = 0, q = k = v = 0, which is an exact
 * no-op on the state.
 *
 * Calls are asynchronous on `stream` (a hipStream_t, NULL = the default
 * stream): they validate the arguments on the host, enqueue the kernels and
 * return.  On a validation failure nothing is enqueued and a negative status
 * is returned.  Values are not checked: non-finite alpha or beta propagate,
 * and alpha < 0 is outside the supported domain (the scan works with
 * log alpha; log alpha is clamped below at -87.3, i.e. alpha < 1.2e-38 acts
 * as that value).
 */
#ifndef GDN_H
#define GDN_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GDN_OK = 0,
    GDN_ERR_NULL = -1,        /* a required pointer is NULL */
    GDN_ERR_SHAPE = -2,       /* a size < 1, or an index would overflow */
    GDN_ERR_UNSUPPORTED = -3, /* Dk/Dv not in {64,128} or chunk != 64 */
    GDN_ERR_WORKSPACE = -4,   /* workspace missing, too small or misaligned */
    GDN_ERR_HIP = -5,         /* a HIP runtime call or kernel launch failed */
    GDN_ERR_ALIGN = -6,       /* a pointer is not 16-byte aligned */
    GDN_ERR_ALIAS = -7        /* out/state_out overlaps an input it may not */
} gdn_status;

/*
 * bf16 path: q, k, v and out hold bf16; alpha, beta and the state are fp32.
 * Products run on bf16 MFMA with fp32 accumulation; the recurrent state stays
 * fp32 across the whole scan.  Uses a workspace cached by the library per
 * device (allocated with hipMalloc on first use and grown when a larger call
 * needs it; a growing call synchronizes the device).  Not safe to call
 * concurrently from several host threads or on several streams at once: use
 * gdn_chunk_forward_ws for that.
 */
int gdn_chunk_forward(const void *q, const void *k, const void *v,
                      const float *alpha, const float *beta, const float *state_in,
                      void *out, float *state_out,
                      int B, int H, int T, int Dk, int Dv, int chunk, void *stream);

/* fp32 path: same contract, q, k, v and out hold fp32 (fp32 MFMA throughout). */
int gdn_chunk_forward_f32(const float *q, const float *k, const float *v,
                          const float *alpha, const float *beta, const float *state_in,
                          float *out, float *state_out,
                          int B, int H, int T, int Dk, int Dv, int chunk, void *stream);

/*
 * Bytes of device workspace the *_ws variants need for this shape
 * (is_bf16 = 1 for the bf16 path, 0 for fp32).  Returns 0 for unsupported
 * or invalid shapes.
 */
size_t gdn_workspace_bytes(int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16);

/*
 * Explicit-workspace variants: identical to the calls above, but use the
 * caller-owned device buffer `ws` (256-byte aligned, at least
 * gdn_workspace_bytes(...) bytes) and allocate nothing.  Concurrent calls
 * are safe when each uses its own workspace.  The workspace holds only
 * intermediate results; its contents on entry do not matter.
 */
int gdn_chunk_forward_ws(const void *q, const void *k, const void *v,
                         const float *alpha, const float *beta, const float *state_in,
                         void *out, float *state_out,
                         int B, int H, int T, int Dk, int Dv, int chunk,
                         void *ws, size_t ws_bytes, void *stream);

int gdn_chunk_forward_f32_ws(const float *q, const float *k, const float *v,
                             const float *alpha, const float *beta, const float *state_in,
                             float *out, float *state_out,
                             int B, int H, int T, int Dk, int Dv, int chunk,
                             void *ws, size_t ws_bytes, void *stream);

/*
 * Scan-group control.  scan_group = chunks per scan group: 0 picks the
 * library's choice (one group when T is at most 64 chunks or when
 * B*H*Dv/16 >= 64 on the bf16 path, >= 512 on the fp32 path; else about
 * sqrt(chunks)), a value >= the number of
 * chunks gives a single sequential scan, and any value in between is used as
 * given (negative counts as 0).  The two calls
 * below take it explicitly: gdn_workspace_bytes_ex sizes the workspace for
 * it (the workspace differs between group sizes), and gdn_chunk_forward_ex
 * is gdn_chunk_forward_ws / gdn_chunk_forward_f32_ws (is_bf16 selects) run
 * with it.  gdn_workspace_bytes(...) equals gdn_workspace_bytes_ex(..., 0).
 */
size_t gdn_workspace_bytes_ex(int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16,
                              int scan_group);

/*
 * Host-only consistency check of the workspace layout (no HIP call): for the
 * path a call with these arguments takes, every region of the workspace
 * (cumulative log decays, per-chunk gate records of key decay factors and
 * chunk decay, -W, U~t, per-chunk states or fused-output operands,
 * pseudo-values, and the grouped scan's transfers,
 * offsets, log decays and entry states) starts 256-byte aligned and spans at
 * least the highest byte the kernels index in it (their index expressions at
 * the largest chunk and group index).  Returns GDN_OK, the 1-based number of
 * the first region that fails, or GDN_ERR_SHAPE / GDN_ERR_UNSUPPORTED.
 */
int gdn_workspace_check(int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16, int scan_group);

/*
 * Allocation-free variant of gdn_chunk_forward (bf16 path), for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  The workspace is an array of
 * GDN_NOALLOC_MAX_WORKSPACE bytes in the library's device code object: each
 * GPU the call runs on holds its own copy until the process ends.  The call
 * makes no hipMalloc, hipFree or other allocating call; on its first use with
 * a device current it looks up that device's copy (hipGetSymbolAddress).
 * Arguments, layouts, validation and results are those of gdn_chunk_forward
 * (bitwise the same outputs).  Shapes whose workspace, gdn_workspace_bytes(...,
 * is_bf16 = 1), exceeds GDN_NOALLOC_MAX_WORKSPACE return GDN_ERR_WORKSPACE
 * before anything is enqueued; one 1280x704 frame (B = 1, T = 3520, H = 16,
 * Dk = Dv = 128: 48.8 MiB) fits.  Every call on a GPU shares that GPU's array:
 * calls that overlap on one GPU (several host threads, or streams not ordered
 * with each other) race and give wrong results.  No part of the array needs to
 * start at zero: every value a call uses was written earlier in the same call
 * (its copies also move a few padding bytes that nothing uses).
 */
#define GDN_NOALLOC_MAX_WORKSPACE ((size_t)64 << 20)
int gdn_chunk_forward_noalloc(const void *q, const void *k, const void *v,
                              const float *alpha, const float *beta, const float *state_in,
                              void *out, float *state_out,
                              int B, int H, int T, int Dk, int Dv, int chunk, void *stream);

/* Chunks per scan group the calls above use for this shape, path (is_bf16)
 * and scan_group (0 for unsupported arguments). */
int gdn_scan_group_size(int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16, int scan_group);

int gdn_chunk_forward_ex(const void *q, const void *k, const void *v,
                         const float *alpha, const float *beta, const float *state_in,
                         void *out, float *state_out,
                         int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16,
                         int scan_group, void *ws, size_t ws_bytes, void *stream);

/*
 * Per-stage timing (measurement aid, same arguments as gdn_chunk_forward_ex):
 * enqueues the path once on `stream`, with every stage launched `reps` times
 * back to back between two HIP events recorded on that stream (a stage's
 * launches are identical re-runs, since a stage only reads the inputs and the
 * previous stages' results), then synchronizes the stream and writes the mean
 * duration of one launch of each stage in milliseconds to stage_ms[0..4]
 * (host memory): [0] WY transform, [1] group transfer maps, [2] scan over
 * groups, [3] chunk states, [4] output.  Stages that do not run for this
 * shape (1 and 2 with a single scan group) report 0.  state_in ==
 * state_out is rejected with GDN_ERR_ALIAS.  The outputs are those of one
 * ordinary call.  Creates and destroys its own events.
 */
int gdn_profile_stages(const void *q, const void *k, const void *v,
                       const float *alpha, const float *beta, const float *state_in,
                       void *out, float *state_out,
                       int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16,
                       int scan_group, void *ws, size_t ws_bytes, int reps, float *stage_ms,
                       void *stream);

/*
 * ---------------------------------------------------------------------------
 * Frame-wise GDN forward: the paper's own form (Section "Frame-wise Gated
 * DeltaNet", equations gdn_combined, appendix_gdn_kv_update and
 * appendix_gdn_kv_compact; the three-phase kernel of Section "Efficient
 * System Co-design" and its Algorithm).  The sequence is F frames of N tokens
 * (T = F * N).  One decay alpha_f per (b, f, h) is shared by the frame's
 * tokens, beta is per token, and all N tokens of a frame update the state at
 * once, with keys multiplied by key_scale (the paper uses 1 / sqrt(Dk * N)):
 *
 *   with K~_f = key_scale K_f ([N][Dk]), B_f = diag(beta_f), H = S^T [Dk][Dv]:
 *     H_f = alpha_f (I - K~_f^T B_f K~_f) H_{f-1} + K~_f^T B_f V_f
 *     o_t = H_f^T q_t  for every token t of frame f (the readout after the
 *                      frame's own update, without normalizer or gate)
 *
 * Layouts as for the token-wise calls, with T = F * N, except
 *   alpha     [B][F][H]          fp32, one decay per frame and head.
 * q, k, v, out, beta, state_in and state_out have the token-wise layouts; the
 * state is H = S^T, fp32, carried in and out exactly as above (state_in ==
 * state_out allowed).  Supported: B, H, F, N >= 1 with B*H <= 65535 and
 * F*N + 64*F + N < 2^31; Dk, Dv in {64, 128}; any N (a frame need not be a
 * multiple of 64 tokens).  key_scale is used as given (a non-finite value
 * propagates).
 *
 * Evaluation: frame summaries G_f = K~^T B K~ and A_f = K~^T B V are formed in
 * parallel over token splits of every frame (fp32 partial sums, reduced in a
 * fixed order, so results are deterministic), the scan over frames runs one
 * wave per (b, h, 16 state columns), and the output is parallel over tokens.
 * The bf16 path rounds beta * k and beta * v, G_f, and the state operand of
 * the products to bf16 (fp32 accumulation; the state itself stays fp32).
 * Asynchronous on `stream`, errors as for the token-wise calls.
 */
int gdn_frame_forward(const void *q, const void *k, const void *v,
                      const float *alpha, const float *beta, const float *state_in,
                      void *out, float *state_out,
                      int B, int H, int F, int N, int Dk, int Dv, float key_scale, void *stream);

int gdn_frame_forward_f32(const float *q, const float *k, const float *v,
                          const float *alpha, const float *beta, const float *state_in,
                          float *out, float *state_out,
                          int B, int H, int F, int N, int Dk, int Dv, float key_scale,
                          void *stream);

/*
 * Token splits per frame used for the summaries (token_splits <= 0: the
 * library's choice, about 512 summary workgroups; otherwise the value given,
 * capped at ceil(N / 64) and reduced so that no split is empty).  0 for
 * unsupported arguments.
 */
int gdn_frame_token_splits(int B, int H, int F, int N, int Dk, int Dv, int token_splits);

/* Workspace bytes gdn_frame_forward_ex needs (0 for unsupported arguments). */
size_t gdn_frame_workspace_bytes(int B, int H, int F, int N, int Dk, int Dv, int is_bf16,
                                 int token_splits);

/*
 * Explicit workspace and token-split count (is_bf16 selects the element type
 * of q, k, v and out).  `ws`: caller-owned device buffer, 256-byte aligned, at
 * least gdn_frame_workspace_bytes(...) bytes; nothing is allocated.
 */
int gdn_frame_forward_ex(const void *q, const void *k, const void *v,
                         const float *alpha, const float *beta, const float *state_in,
                         void *out, float *state_out,
                         int B, int H, int F, int N, int Dk, int Dv, float key_scale,
                         int is_bf16, int token_splits, void *ws, size_t ws_bytes, void *stream);

/*
 * Per-stage timing of the frame-wise path (measurement aid, arguments as
 * gdn_frame_forward_ex): each of the four stages is launched `reps` times back
 * to back between two events; stage_ms[0..3] (host memory) receives the mean
 * duration of one launch of [0] frame summaries, [1] reduction over splits,
 * [2] scan over frames, [3] output.  state_in == state_out is rejected with
 * GDN_ERR_ALIAS.  Synchronizes the stream.
 */
int gdn_frame_profile_stages(const void *q, const void *k, const void *v,
                             const float *alpha, const float *beta, const float *state_in,
                             void *out, float *state_out,
                             int B, int H, int F, int N, int Dk, int Dv, float key_scale,
                             int is_bf16, int token_splits, void *ws, size_t ws_bytes, int reps,
                             float *stage_ms, void *stream);

/*
 * Frame-wise forward with the normalizer state and the normalized readout
 * (Section "Frame-wise Gated DeltaNet": equation appendix_gdn_z_update /
 * appendix_gdn_z_compact for the state, equation appendix_gdn_readout for the
 * readout; no rotary embedding on this path, so rotated and unrotated keys and
 * queries coincide).  Beside H, a vector state z = S^z of length Dk per (b, h)
 * is carried from the keys alone:
 *
 *     z_f = alpha_f (I - K~_f^T B_f K~_f) z_{f-1} + K~_f^T beta_f
 *     o_t = (H_f^T q_t) / (z_f . q_t + eps)      for every token t of frame f
 *
 * (eps: the paper uses 1e-6).  Everything else is as gdn_frame_forward;
 * in addition
 *   z_in   [B][H][Dk]   fp32 device pointer or NULL (zero state)
 *   z_out  [B][H][Dk]   fp32 device pointer or NULL (terminal z dropped)
 * z_in == z_out (in place) is allowed; z_out may not overlap any other input
 * or output.  The denominator is not checked: the paper's non-negative
 * feature maps keep it positive, other inputs can make it vanish.
 * is_bf16 selects the element type of q, k, v and out.  On the bf16 path z
 * enters the products rounded to bf16 (as H does), the states stay fp32.
 * gdn_frame_forward_norm uses the library-cached workspace;
 * gdn_frame_forward_norm_ex a caller-owned one of gdn_frame_workspace_bytes
 * (the same size as for the un-normalized call) and an explicit token-split
 * count; gdn_frame_profile_stages_norm times the four stages like
 * gdn_frame_profile_stages (rejecting state_in == state_out and
 * z_in == z_out).
 */
int gdn_frame_forward_norm(const void *q, const void *k, const void *v,
                           const float *alpha, const float *beta, const float *state_in,
                           const float *z_in, void *out, float *state_out, float *z_out,
                           int B, int H, int F, int N, int Dk, int Dv, float key_scale, float eps,
                           int is_bf16, void *stream);

int gdn_frame_forward_norm_ex(const void *q, const void *k, const void *v,
                              const float *alpha, const float *beta, const float *state_in,
                              const float *z_in, void *out, float *state_out, float *z_out,
                              int B, int H, int F, int N, int Dk, int Dv, float key_scale, float eps,
                              int is_bf16, int token_splits, void *ws, size_t ws_bytes,
                              void *stream);

int gdn_frame_profile_stages_norm(const void *q, const void *k, const void *v,
                                  const float *alpha, const float *beta, const float *state_in,
                                  const float *z_in, void *out, float *state_out, float *z_out,
                                  int B, int H, int F, int N, int Dk, int Dv, float key_scale,
                                  float eps, int is_bf16, int token_splits, void *ws,
                                  size_t ws_bytes, int reps, float *stage_ms, void *stream);

/*
 * Bidirectional frame-wise forward (Section "Efficient System Co-design",
 * paragraph on the GDN kernel, Algorithm Phase B: a forward scan from the
 * cached state plus a backward scan within the call from a zero state, the
 * two histories added before the readout).  With U_f the frame update of
 * gdn_frame_forward (U_f(X) = alpha_f (X - G_f X) + A_f):
 *
 *     H_f  = U_f(H_{f-1})          forward, from state_in
 *     Hb_{F-1} = 0,  Hb_{f-1} = U_f(Hb_f)   backward over the later frames
 *     o_t  = (H_f + Hb_f)^T q_t    for every token t of frame f
 *
 * normalized != 0 carries z and zb the same way (the backward one from zero)
 * and divides by (z_f + zb_f) . q_t + eps, as gdn_frame_forward_norm;
 * normalized == 0 ignores z_in, z_out and eps.  state_out (and z_out) receive
 * the forward terminal state only, the one a cache carries to the next call;
 * the backward histories live in the workspace for the duration of the call.
 * F == 1 gives the unidirectional result.  Arguments, layouts, aliasing rules
 * and errors as gdn_frame_forward_norm; the same workspace size
 * (gdn_frame_workspace_bytes) serves every variant.  gdn_frame_forward_bidir
 * uses the library-cached workspace, gdn_frame_forward_bidir_ex a caller-owned
 * one and an explicit token-split count; gdn_frame_profile_stages_bidir times
 * the four stages as gdn_frame_profile_stages (the scan stage includes the
 * backward sweep).
 */
int gdn_frame_forward_bidir(const void *q, const void *k, const void *v,
                            const float *alpha, const float *beta, const float *state_in,
                            const float *z_in, void *out, float *state_out, float *z_out,
                            int B, int H, int F, int N, int Dk, int Dv, float key_scale, float eps,
                            int is_bf16, int normalized, void *stream);

int gdn_frame_forward_bidir_ex(const void *q, const void *k, const void *v,
                               const float *alpha, const float *beta, const float *state_in,
                               const float *z_in, void *out, float *state_out, float *z_out,
                               int B, int H, int F, int N, int Dk, int Dv, float key_scale,
                               float eps, int is_bf16, int normalized, int token_splits, void *ws,
                               size_t ws_bytes, void *stream);

int gdn_frame_profile_stages_bidir(const void *q, const void *k, const void *v,
                                   const float *alpha, const float *beta, const float *state_in,
                                   const float *z_in, void *out, float *state_out, float *z_out,
                                   int B, int H, int F, int N, int Dk, int Dv, float key_scale,
                                   float eps, int is_bf16, int normalized, int token_splits,
                                   void *ws, size_t ws_bytes, int reps, float *stage_ms,
                                   void *stream);

/*
 * The fused GDN operator around the frame-wise normalized recurrence (appendix
 * on the GDN block: subsection "Attention features" for the feature maps and
 * the key rescale; subsection "Frame-wise delta-rule update", equations
 * appendix_gdn_kv_update and appendix_gdn_z_update; subsection "Normalized
 * readout and output projection", equations appendix_gdn_readout and
 * appendix_gdn_output; Algorithm alg:gdn-kernel).  bf16 here; the _f32 calls
 * below are the fp32 mode.  Per token n and head h, from the raw projections
 * q_n = q_raw[b][n][h], k_n (length Dk):
 *
 *   r(x)  = gain o x / sqrt(mean_i x_i^2 + rms_eps)       (RMSNorm over Dk)
 *   q~ = ReLU(r_q(q_n)),   k~ = key_scale ReLU(r_k(k_n))   (unrotated features)
 *   q^ = R_n q~,           k^ = R_n k~                     (3D RoPE)
 *   H_f = alpha_f (H - K^_f^T B_f K^_f H) + K^_f^T B_f V_f          (rotated keys)
 *   z_f = alpha_f (z - K~_f^T B_f K~_f z) + K~_f^T beta_f           (unrotated keys)
 *   y_n = (H_f^T q^_n) / (z_f . q~_n + eps)
 *   out_n = W_o[h] (SiLU(gate_n) o y_n),   SiLU(x) = x / (1 + e^-x)
 *
 * R_n rotates channel pair (2i, 2i+1) by theta_i = rope_freq[i] * c_i(n):
 * (x_2i, x_2i+1) -> (x_2i cos - x_2i+1 sin, x_2i sin + x_2i+1 cos), with c_i
 * the coordinate of token n = f N + s of the call along rope_axis[i]: 0 the
 * time t0 + f, 1 the latent row s / lat_w, any other value the latent column
 * s % lat_w.  With bidirectional != 0 both states get the backward histories
 * of gdn_frame_forward_bidir before the readout.
 *
 *   q_raw, k_raw  [B][T][H][Dk]   bf16     gate  [B][T][H][Dv]  bf16 (before the SiLU)
 *   v, out        [B][T][H][Dv]   bf16     w_o   [H][Dv][Dv]    bf16, row = output channel
 *   gain_q, gain_k [H][Dk]  fp32           rope_freq [Dk/2] fp32 (radians per unit)
 *   rope_axis [Dk/2] int32                 alpha, beta, states: as gdn_frame_forward_norm
 *   lat_w >= 1 (tokens per latent row), t0 (time coordinate of frame 0)
 *
 * All pointers are device pointers (16-byte aligned); gate, w_o, the gains
 * and the RoPE arrays are required.  Outputs may not overlap any input;
 * state_in == state_out and z_in == z_out are allowed.  The bf16 path rounds
 * the features, the gated readout and the products' operands to bf16 (fp32
 * accumulation); the sines and cosines are the GPU's hardware ones, on angles
 * reduced to one turn.
 * gdn_frame_forward_fused uses the library-cached workspace,
 * gdn_frame_forward_fused_ex a caller-owned one of gdn_frame_workspace_bytes
 * (is_bf16 = 1) and an explicit token-split count; gdn_frame_profile_stages_fused
 * times the four stages (its last stage is the fused output).  Errors as the
 * other frame-wise calls; a missing prologue/epilogue input is GDN_ERR_NULL,
 * lat_w < 1 GDN_ERR_SHAPE.
 */
int gdn_frame_forward_fused(const void *q_raw, const void *k_raw, const void *v, const void *gate,
                            const void *w_o, const float *alpha, const float *beta,
                            const float *gain_q, const float *gain_k, const float *rope_freq,
                            const int *rope_axis, const float *state_in, const float *z_in,
                            void *out, float *state_out, float *z_out,
                            int B, int H, int F, int N, int Dk, int Dv, int lat_w, int t0,
                            float key_scale, float rms_eps, float eps, int bidirectional,
                            void *stream);

int gdn_frame_forward_fused_ex(const void *q_raw, const void *k_raw, const void *v, const void *gate,
                               const void *w_o, const float *alpha, const float *beta,
                               const float *gain_q, const float *gain_k, const float *rope_freq,
                               const int *rope_axis, const float *state_in, const float *z_in,
                               void *out, float *state_out, float *z_out,
                               int B, int H, int F, int N, int Dk, int Dv, int lat_w, int t0,
                               float key_scale, float rms_eps, float eps, int bidirectional,
                               int token_splits, void *ws, size_t ws_bytes, void *stream);

int gdn_frame_profile_stages_fused(const void *q_raw, const void *k_raw, const void *v,
                                   const void *gate, const void *w_o, const float *alpha,
                                   const float *beta, const float *gain_q, const float *gain_k,
                                   const float *rope_freq, const int *rope_axis,
                                   const float *state_in, const float *z_in, void *out,
                                   float *state_out, float *z_out, int B, int H, int F, int N,
                                   int Dk, int Dv, int lat_w, int t0, float key_scale,
                                   float rms_eps, float eps, int bidirectional, int token_splits,
                                   void *ws, size_t ws_bytes, int reps, float *stage_ms,
                                   void *stream);

/*
 * The fused operator in fp32 (the paper's "ieee" precision mode, appendix "GDN
 * Kernel Details", "Precision modes"): the same computation as
 * gdn_frame_forward_fused with q_raw, k_raw, v, gate, w_o and out in fp32 and
 * every feature, product and readout in fp32 (no bf16 rounding anywhere; the
 * rotation angles in fp64 with accurate sines and cosines).  Arguments,
 * layouts, aliasing rules and errors as the bf16 calls.  The workspace also
 * holds the four feature maps and the gated readout (about
 * 4 B T H (4 Dk + Dv) bytes on top): size it with
 * gdn_frame_fused_workspace_bytes(..., is_bf16 = 0, ...).
 * gdn_frame_profile_stages_fused_f32 times four stages: features and
 * summaries, reduction, scan, output and projection.
 */
int gdn_frame_forward_fused_f32(const float *q_raw, const float *k_raw, const float *v,
                                const float *gate, const float *w_o, const float *alpha,
                                const float *beta, const float *gain_q, const float *gain_k,
                                const float *rope_freq, const int *rope_axis,
                                const float *state_in, const float *z_in, float *out,
                                float *state_out, float *z_out, int B, int H, int F, int N,
                                int Dk, int Dv, int lat_w, int t0, float key_scale,
                                float rms_eps, float eps, int bidirectional, void *stream);

int gdn_frame_forward_fused_f32_ex(const float *q_raw, const float *k_raw, const float *v,
                                   const float *gate, const float *w_o, const float *alpha,
                                   const float *beta, const float *gain_q, const float *gain_k,
                                   const float *rope_freq, const int *rope_axis,
                                   const float *state_in, const float *z_in, float *out,
                                   float *state_out, float *z_out, int B, int H, int F, int N,
                                   int Dk, int Dv, int lat_w, int t0, float key_scale,
                                   float rms_eps, float eps, int bidirectional, int token_splits,
                                   void *ws, size_t ws_bytes, void *stream);

int gdn_frame_profile_stages_fused_f32(const float *q_raw, const float *k_raw, const float *v,
                                       const float *gate, const float *w_o, const float *alpha,
                                       const float *beta, const float *gain_q, const float *gain_k,
                                       const float *rope_freq, const int *rope_axis,
                                       const float *state_in, const float *z_in, float *out,
                                       float *state_out, float *z_out, int B, int H, int F, int N,
                                       int Dk, int Dv, int lat_w, int t0, float key_scale,
                                       float rms_eps, float eps, int bidirectional,
                                       int token_splits, void *ws, size_t ws_bytes, int reps,
                                       float *stage_ms, void *stream);

/* Workspace bytes the fused operator's _ex calls need (is_bf16 = 1: equal to
 * gdn_frame_workspace_bytes; 0 for unsupported arguments). */
size_t gdn_frame_fused_workspace_bytes(int B, int H, int F, int N, int Dk, int Dv, int is_bf16,
                                       int token_splits);

/* Static, human-readable text for a status code. */
const char *gdn_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* GDN_H */
