// Frame-wise GDN forward (the paper's own form): Section "Frame-wise Gated
// DeltaNet", equations gdn_combined, appendix_gdn_kv_update and
// appendix_gdn_kv_compact; Section "Efficient System Co-design", paragraph on
// the GDN kernel, and its Algorithm (Phase A frame summaries, Phase B scan
// over frames, Phase C output).
//
// One decay alpha_f per frame and head is shared by the frame's N tokens,
// which all write at once; beta is per token; the keys enter the recurrence
// multiplied by key_scale (the paper uses 1 / sqrt(D N)).  In the H = S^T
// orientation ([Dk][Dv] per head), with K~ = key_scale K and B_f = diag(beta):
//     G_f = K~_f^T B_f K~_f                 (Dk x Dk)   Phase A
//     A_f = K~_f^T B_f V_f                  (Dk x Dv)   Phase A
//     H_f = alpha_f (H_{f-1} - G_f H_{f-1}) + A_f       Phase B
//     O_f = Q_f H_f                                     Phase C
// (P_f = I - G_f: the identity part is applied exactly in fp32 and only the
// correction G_f H_{f-1} goes through the MFMAs.)
//
// Kernels, E = bf16 bits or fp32 storage, fp32 accumulation everywhere:
//   gdn_frame_summary_kernel  (token split s, frame f, head): G and A over the
//       split's tokens, 64-token blocks streamed through an LDS ring by loader
//       waves; the final G fragments and A tiles with a single split, else
//       fp32 partial tiles.
//   gdn_frame_reduce_kernel   sums the NS splits' partials and applies the
//       key scale: G as ready-made MFMA operand fragments (E), A as fp32
//       accumulator tiles.
//   gdn_frame_scan_kernel     one wave per (head, 16 state columns): H_f for
//       every frame in turn, written as the output kernel's operand
//       fragments (E), and the terminal state; in the bidirectional form a
//       backward sweep first, whose histories are added to the H_f written.
//   gdn_frame_output_kernel   a run of 16-token tiles of one frame per
//       workgroup: O^T = H_f^T Q^T.
// The normalizer (NORM variants) rides along as one more 16-column state
// tile.  The fused operator (FUSED variants, bf16) forms the key features in
// the summary kernel, carries the normalizer on its own Gram matrix of the
// unrotated keys, and ends in gdn_frame_output_fused_kernel (query features,
// gate and per-head projection).
//
// Tile layouts (see gdn_device.h for the lane conventions).  Accumulator
// tiles over the Dk rows are in P32 order: row tile r = 2 m + a holds rows
// 32 m + p32_row(a, i), so lane (li, lg) holds rows 32 m + 8 lg + 4 a + q.
// G tiles are in P32 order along the columns too.  Because G is symmetric,
// the pair of partial tiles (r = 2 kb, c = t), (r = 2 kb + 1, c = t) is, lane
// by lane, the A operand fragment of row tile t of G over the k block kb.
#pragma once

#include <type_traits>

#include "gdn_device.h"

namespace gdn {

// Rotation angles are formed in turns (the pair's frequency / 2 pi times the
// token's coordinate on its axis) and reduced to [-1/2, 1/2] before the
// hardware sine and cosine, whose input is in turns and whose accuracy holds
// only over a bounded range; so long time coordinates stay accurate up to the
// fp32 rounding of the angle itself.
constexpr float kInvTwoPi = 0.15915494309189535f;

template <class E> struct FrameParams {
    const E *q, *k, *v;          // [B][T][H][Dk] / [Dv], T = F * N
    const float *alpha;          // [B][F][H]
    const float *beta;           // [B][T][H]
    const float *state_in;       // [B][H][Dk][Dv] or null (zero)
    E *out;                      // [B][T][H][Dv]
    float *state_out;            // [B][H][Dk][Dv] or null
    int B, H, F, N;
    int NS, NBT;                 // token splits per frame, tokens per split (a multiple of 64)
    int OB, OTPW;                // output workgroups per frame, 16-token tiles per workgroup
    float key_scale;
    // normalizer (the kernels' NORM variant): z = S^z as one more state
    // column tile, written by value columns of ones, so that each of its 16
    // columns holds z; NJ = Dv / 16 + NORM column tiles below
    const float *z_in;           // [B][H][Dk] or null (zero)
    float *z_out;                // [B][H][Dk] or null
    float eps;
    float *PG;                   // [B*H][F][NS][Dk/16][Dk/16][64][4]  partial G tiles
    float *PA;                   // [B*H][F][NS][Dk/16][NJ][64][4]     partial A tiles
    E *Gf;                       // [B*H][F][Dk/16][Dk/32][64][8]      G operand fragments
    float *Af;                   // [B*H][F][Dk/16][NJ][64][4]         A tiles
    E *Hf;                       // [B*H][F][NJ][Dk/32][64][8]         H_f operand fragments
    float *Hb;                   // [B*H][F][NJ][Dk/16][64][4]         backward histories (bidirectional)
    // fused operator (the FUSED variants): raw projections in q and k, the
    // feature maps formed on load; the normalizer recurrence takes its own
    // Gram matrix of the unrotated keys
    E *Gzf;                      // [B*H][F][Dk/16][Dk/32][64][8]      unrotated-key G fragments
    float *PGz;                  // [B*H][F][NS][Dk/16][Dk/16][64][4]  its partial tiles
    const E *gate;               // [B][T][H][Dv]  output gate before the SiLU
    const E *w_o;                // [H][Dv][Dv]    per-head output projection (row = output channel)
    const float *gain_q, *gain_k;  // [H][Dk]      RMSNorm gains
    const float *rope_freq;      // [Dk/2]         angle per coordinate unit of channel pair i
    const int *rope_axis;        // [Dk/2]         its coordinate: 0 time, 1 latent row, else latent column
    float rms_eps, feat_scale;   // RMSNorm epsilon; key scale applied to the key features
    int lat_w, t0;               // tokens per latent row; time coordinate of frame 0
    // the fused operator in fp32: its feature maps and gated readout in the
    // workspace, and which summaries a summary launch stores
    float *fqt, *fqh, *fkt, *fkh;  // [B][T][H][Dk]  q~, q^, k~, k^
    float *ybuf;                 // [B][T][H][Dv]  SiLU(gate) o y
    int sum_mode;                // 0 all; 1 all but the normalizer tile; 2 all but the A tiles
};

// A fragment of ones: as the B operand, a 16-column tile whose every column is
// a value column of ones, so every column of the product K~^T B [1 .. 1] is
// K~^T beta.
template <class E> __device__ __forceinline__ typename Tr<E>::frag ones_frag();
template <> __device__ __forceinline__ Tr<uint16_t>::frag ones_frag<uint16_t>() {
    const uint32_t x = 0x3f803f80u;                             // two bf16 ones
    return Tr<uint16_t>::frag{x, x, x, x};
}
template <> __device__ __forceinline__ Tr<float>::frag ones_frag<float>() {
    return Tr<float>::frag{1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f, 1.f};
}

// Grids of per_unit workgroups per unit with all workgroups of one unit on
// one XCD (blocks are dealt to the 8 XCDs round robin: id = 8 y + x runs on
// XCD x), so the data they share is fetched into one L2.
inline unsigned xcd_blocks(long long units, int per_unit) {
    return 8u * (unsigned)per_unit * (unsigned)((units + 7) / 8);
}
__device__ __forceinline__ void xcd_unit(int id, int per_unit, int &unit, int &sub) {
    const int x = id & 7, y = id >> 3;
    sub = y % per_unit;
    unit = 8 * (y / per_unit) + x;
}

// LDS ring of the summary kernel: DEPTH slots, each one 64-token block of
// raw keys, raw values and the block's 64 betas (FUSED: the raw keys become
// the unrotated features in place, and a second key area takes the rotated
// ones).  A 64-row tile with R
// 16-byte chunks per row is stored in groups of four rows: chunk c of row r
// sits at chunk position 4 R (r / 4) + 16 (c / 4) + 4 (r % 4) + c % 4.  A 1 KB
// copy then reads contiguous runs of at least 256 bytes (4 rows of 16 chunks,
// or whole rows when a row is shorter), and the transposed operand reads of a
// fragment differ from one fragment to the next by a constant offset.
template <class E, int DK, int DV, bool FUSED = false> struct FrameSumLds {
    static constexpr int KB_ = 64 * DK * (int)sizeof(E), VB_ = 64 * DV * (int)sizeof(E);
    static constexpr int KH_ = FUSED ? KB_ : 0;                  // rotated key features (FUSED)
    static constexpr int SLOT = KB_ + VB_ + KH_ + 256;
    static constexpr int NCK = KB_ / 1024, NCV = VB_ / 1024;   // 1 KB copies per block
    static constexpr int CAP = 160 * 1024;
    static constexpr int DL = (CAP - (FUSED ? 1024 : 0)) / SLOT;
    // loaders 0, 1 (halves of the key copies, 0 also the betas) and 2, 3
    // (halves of the value copies) wait with DEPTH - 2 younger blocks in
    // flight: vmcnt <= 63
    static constexpr int PER = NCK / 2 + 1 > NCV / 2 ? NCK / 2 + 1 : NCV / 2;
    static constexpr int DVM = 2 + 63 / PER;
    static constexpr int D0 = DL < DVM ? DL : DVM;
    static constexpr int DEPTH = D0 < 6 ? D0 : 6;
    static constexpr size_t oK = 0, oV = KB_, oB = KB_ + VB_, oKh = KB_ + VB_ + 256;
    // FUSED: after the ring, 1 KB that takes the copies issued past the last
    // block (their slot is being transformed in place)
    static constexpr size_t oDm = (size_t)DEPTH * SLOT;
    static constexpr size_t bytes = oDm + (FUSED ? 1024 : 0);
    static_assert(!FUSED || DEPTH >= 3, "the fused ring holds a block in use, one being formed and one loading");
    // fused loaders wait for their own copies (a quarter of the key and value
    // copies, loader 0 also the betas) with DEPTH - 2 younger blocks in flight
    static_assert(!FUSED || (DEPTH - 2) * (NCK / 4 + NCV / 4 + 1) <= 63, "fused waits within vmcnt");
    static_assert(DEPTH >= 2, "summary ring needs two slots");
    static_assert(KB_ % 2048 == 0 && VB_ % 2048 == 0, "whole 1 KB copies, two loaders each");
};

// Element offset of (row, col) in a grouped 64-row tile of R chunks per row.
template <class E, int R> __device__ __forceinline__ int gm_at(int row, int col) {
    constexpr int EPC = 16 / (int)sizeof(E);                      // elements per chunk
    const int c = col / EPC;
    return EPC * (4 * R * (row >> 2) + 16 * (c >> 2) + 4 * (row & 3) + (c & 3)) + col % EPC;
}

// Row and chunk that lane l of 1 KB copy ci moves into a grouped tile of R
// chunks per row (chunk position 64 ci + l).
template <int R> __device__ __forceinline__ void gm_src(int ci, int l, int &row, int &chunk) {
    const int pos = 64 * ci + l, g = pos / (4 * R), w = pos % (4 * R);
    row = 4 * g + ((w & 15) >> 2);
    chunk = 4 * (w >> 4) + (w & 3);
}

// Operand fragment over a 32-row k block of a grouped LDS tile: the same
// values as tr_frag on the row-major tile.
template <class E, int R>
__device__ __forceinline__ typename Tr<E>::frag tr_frag_gm(const E *M, int row0, int colbase, bool p32, int a,
                                                           int li, int lg) {
    if constexpr (sizeof(E) == 2) {
        typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
        const int row = row0 + 8 * lg + (li >> 2);
        const int col = p32 ? colbase + 8 * (li & 3) + 4 * a : colbase + 4 * (li & 3);
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(M + gm_at<E, R>(row, col)));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(M + gm_at<E, R>(row + 4, col)));
        return Tr<E>::cat(__builtin_bit_cast(u32x2, lo), __builtin_bit_cast(u32x2, hi));
    } else {
        const int col = p32 ? colbase + p32_row(a, li) : colbase + li;
        typename Tr<E>::frag f;
#pragma unroll
        for (int q = 0; q < 8; ++q) f[q] = M[gm_at<E, R>(row0 + 8 * lg + q, col)];
        return f;
    }
}

// The 8 k-slots of a lane's fragment times 8 per-slot scales.
__device__ __forceinline__ Tr<uint16_t>::frag scale_frag(Tr<uint16_t>::frag x, const float (&b)[8]) {
    Tr<uint16_t>::frag y;
#pragma unroll
    for (int d = 0; d < 4; ++d)
        y[d] = pack_bf16x2(__uint_as_float(x[d] << 16) * b[2 * d], __uint_as_float(x[d] & 0xffff0000u) * b[2 * d + 1]);
    return y;
}
__device__ __forceinline__ Tr<float>::frag scale_frag(Tr<float>::frag x, const float (&b)[8]) {
#pragma unroll
    for (int q = 0; q < 8; ++q) x[q] *= b[q];
    return x;
}

// Sum over aligned groups of R lanes (R = 8 or 16), every lane of a group
// receiving the group's sum, with DPP lane moves (no LDS traffic): swaps
// within quads, then the mirror within 8 lanes, then within 16.
template <int R> __device__ __forceinline__ float group_sum(float x) {
    static_assert(R == 8 || R == 16, "group of 8 or 16 lanes");
    auto dpp = [](float v, auto ctrl) {
        return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), decltype(ctrl)::value, 0xf, 0xf, false));
    };
    x += dpp(x, std::integral_constant<int, 0xB1>{});                  // quad_perm [1, 0, 3, 2]
    x += dpp(x, std::integral_constant<int, 0x4E>{});                  // quad_perm [2, 3, 0, 1]
    x += dpp(x, std::integral_constant<int, 0x141>{});                 // row_half_mirror
    if constexpr (R == 16) x += dpp(x, std::integral_constant<int, 0x140>{});   // row_mirror
    return x;
}

// Phase A.  Workgroup (token split s, frame f, head): [G | A] over the split's
// tokens (G = K^T B K with P32 rows and columns, A = K^T B V with P32 rows),
// with 8 compute waves and 4 loader waves.  The loaders copy 64-token blocks
// of raw K, V and beta into the LDS ring (asynchronous global->LDS copies,
// DEPTH - 1 blocks ahead).  Compute wave w < 4 accumulates G, wave 4 + w A:
// P32 row pair kb = w % (Dk / 32), i.e. row tiles 2 kb and 2 kb + 1, and a
// share of the column tiles.  beta multiplies the K^T operand fragments in
// registers (zero for tokens past the split).
// With a single split the workgroup writes G's operand fragments (key scale
// squared) and A's tiles (key scale) in their final form: the pair of row
// tiles (2 kb, 2 kb + 1) of G column tile t is, lane by lane, fragment (t, kb).
// With several splits it writes fp32 partial tiles for the reduction.
// FUSED (the whole operator; bf16): the keys arrive raw.  A three-stage ring:
// while the compute waves multiply block i, each loader wave waits for its
// own copies of block i + 1 -- the key rows 16 ld .. 16 ld + 15 and a share
// of the values -- and turns those rows into the unrotated features
// k~ = key_scale ReLU(gain o k / rms(k)) in place and their rotations
// k^ = R k~ (3D RoPE) into a second area of the slot (Dk / 8 lanes per row,
// the row's sum of squares reduced across them); the next barrier hands both
// over.  G and A take k^; four more compute waves accumulate the unrotated
// Gram matrix K~^T B K~ and K~^T beta for the normalizer.  The key scale is
// then already in the features.
constexpr int kSumCompute = 8, kSumLoaders = 4;
template <bool FUSED> constexpr int sum_threads() { return (kSumCompute + (FUSED ? 4 : 0) + kSumLoaders) * 64; }

template <class E, int DK, int DV, bool NORM, bool FUSED = false>
__global__ __launch_bounds__(sum_threads<FUSED>()) void gdn_frame_summary_kernel(FrameParams<E> p) {
    static_assert(!FUSED || (NORM && sizeof(E) == 2), "the fused operator is normalized and bf16");
    using L = FrameSumLds<E, DK, DV, FUSED>;
    using TR = Tr<E>;
    using frag = typename TR::frag;
    constexpr int D = L::DEPTH;
    constexpr int ESZ = (int)sizeof(E);
    constexpr int RK = DK * ESZ / 16, RV = DV * ESZ / 16;             // chunks per tile row
    constexpr int NCK2 = L::NCK / 2, NCV2 = L::NCV / 2;
    constexpr int NR = DK / 16, NP = NR / 2, KBN = DK / 32;           // row tiles, row pairs
    constexpr int NCG = DK / 16, NCA = DV / 16;                       // column tiles of G, A
    constexpr int NJA = NCA + NORM;                                   // A tiles incl. the normalizer
    constexpr int SUB = 4 / NP;                                       // column shares per pair
    constexpr int CPG = NCG / SUB, CPA = NCA / SUB;                   // column tiles per wave
    extern __shared__ __align__(16) unsigned char smem[];
    const int u = blockIdx.x;
    if (u >= p.NS * p.F * p.B * p.H) return;
    const int s = u % p.NS, rest = u / p.NS, f = rest % p.F, bh = rest / p.F;
    const int b = bh / p.H, h = bh - b * p.H;
    const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), l = tid & 63, li = l & 15,
              lg = l >> 4;
    const size_t T = (size_t)p.F * p.N;
    const int t_lo = f * p.N + s * p.NBT;
    const int t_hi = min(f * p.N + p.N, t_lo + p.NBT);
    const int nb = (t_hi - t_lo + 63) / 64;
    const size_t row_b = (size_t)b * T;
    auto slot = [&](int i) { return smem + (size_t)(i % D) * L::SLOT; };
    constexpr int NCOMP = kSumCompute + (FUSED ? 4 : 0);

    if constexpr (FUSED) if (w >= NCOMP) {
        // ---------------- loader waves (FUSED) ----------------
        const int ld = w - NCOMP;
        constexpr int CK = L::NCK / 4, CV = L::NCV / 4;               // copies per loader and block
        static_assert(L::NCK % 4 == 0 && L::NCV % 4 == 0, "whole copies per loader");
        // block ii's copies by this loader (past the last block: the last
        // block's again, into the dummy area, so that every iteration issues
        // the same number of copies and the waits count right)
        auto issue = [&](int ii) {
            const int i = min(ii, nb - 1);
            const bool dummy = ii >= nb;
            const int t0 = t_lo + 64 * i, rmax = t_hi - 1 - t0;
            const size_t row0 = (row_b + t0) * p.H + h;
            unsigned char *sl = dummy ? smem + L::oDm : slot(i);
            const size_t stepc = dummy ? 0 : 1024;
            const char *kb_ = (const char *)(p.k + row0 * DK);
            const unsigned krs = (unsigned)(p.H * DK * ESZ);
#pragma unroll
            for (int j = 0; j < CK; ++j) {
                const int ci = ld * CK + j;
                int r, c;
                gm_src<RK>(ci, l, r, c);
                __builtin_amdgcn_global_load_lds(
                    (const void *)(kb_ + (unsigned)min(r, rmax) * krs + 16u * (unsigned)c),
                    (__attribute__((address_space(3))) void *)(sl + (dummy ? 0 : L::oK) + stepc * ci), 16, 0, 0);
            }
            const char *vb_ = (const char *)(p.v + row0 * DV);
            const unsigned vrs = (unsigned)(p.H * DV * ESZ);
#pragma unroll
            for (int j = 0; j < CV; ++j) {
                const int ci = ld * CV + j;
                int r, c;
                gm_src<RV>(ci, l, r, c);
                __builtin_amdgcn_global_load_lds(
                    (const void *)(vb_ + (unsigned)min(r, rmax) * vrs + 16u * (unsigned)c),
                    (__attribute__((address_space(3))) void *)(sl + (dummy ? 0 : L::oV) + stepc * ci), 16, 0, 0);
            }
            if (ld == 0) {
                const char *bb = (const char *)(p.beta + row0);
                __builtin_amdgcn_global_load_lds(
                    (const void *)(bb + (unsigned)min(l, rmax) * (unsigned)(4 * p.H)),
                    (__attribute__((address_space(3))) void *)(sl + (dummy ? 0 : L::oB)), 4, 0, 0);
            }
        };
        // this loader's copies of the next block have landed once at most
        // D - 2 younger blocks are in flight
        auto wait_next = [&]() {
            if (ld == 0) wait_vmcnt<(D - 2) * (CK + CV + 1)>();
            else wait_vmcnt<(D - 2) * (CK + CV)>();
        };
        // this lane's channels 8 cc .. 8 cc + 7 (pairs 4 cc ..): gains,
        // pair frequencies and axes
        const int cc = l % RK;
        float gk[8], wt[4], wy[4], wx[4];        // per pair: turns per unit of time, row, column
#pragma unroll
        for (int q = 0; q < 8; ++q) gk[q] = p.gain_k[h * DK + 8 * cc + q];
#pragma unroll
        for (int d = 0; d < 4; ++d) {
            const float fq = p.rope_freq[4 * cc + d] * kInvTwoPi;   // turns per unit
            const int a = p.rope_axis[4 * cc + d];
            wt[d] = a == 0 ? fq : 0.f;
            wy[d] = a == 1 ? fq : 0.f;
            wx[d] = (a != 0 && a != 1) ? fq : 0.f;
        }
        const float ct = (float)(p.t0 + f);
        // rows 16 ld .. 16 ld + 15 of block i, 64 / RK rows per pass; all of
        // the wave's reads are issued before its first write
        auto transform = [&](int i) {
            constexpr int NPASS = 16 * RK / 64;
            unsigned char *sl = slot(i);
            E *sK = (E *)(sl + L::oK), *sKh = (E *)(sl + L::oKh);
            const int tok0 = t_lo + 64 * i, rmax = t_hi - 1 - tok0;
            u32x4 raws[NPASS];
#pragma unroll
            for (int ps = 0; ps < NPASS; ++ps)
                raws[ps] = *(const u32x4 *)(sK + gm_at<E, RK>(16 * ld + ps * (64 / RK) + l / RK, 8 * cc));
#pragma unroll
            for (int ps = 0; ps < NPASS; ++ps) {
                const int r = 16 * ld + ps * (64 / RK) + l / RK;
                E *src = sK + gm_at<E, RK>(r, 8 * cc);
                const u32x4 raw = raws[ps];
                float x[8];
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    x[2 * d] = __uint_as_float(raw[d] << 16);
                    x[2 * d + 1] = __uint_as_float(raw[d] & 0xffff0000u);
                }
                float ss = 0.f;
#pragma unroll
                for (int q = 0; q < 8; ++q) ss += x[q] * x[q];
                ss = group_sum<RK>(ss);
                const float inv = rsqrtf(ss * (1.f / DK) + p.rms_eps);
                // the token in this row (rows past the split repeat its last
                // one) and its latent row and column
                const int s_in = tok0 + min(r, rmax) - f * p.N;
                const int yc = s_in / p.lat_w;
                const float cy = (float)yc, cx = (float)(s_in - yc * p.lat_w);
                u32x4 ft, fh;
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    const float x0 = p.feat_scale * fmaxf(gk[2 * d] * x[2 * d] * inv, 0.f);
                    const float x1 = p.feat_scale * fmaxf(gk[2 * d + 1] * x[2 * d + 1] * inv, 0.f);
                    float rv = wt[d] * ct + wy[d] * cy + wx[d] * cx;
                    rv -= rintf(rv);
                    const float sn = __builtin_amdgcn_sinf(rv), cs = __builtin_amdgcn_cosf(rv);
                    ft[d] = pack_bf16x2(x0, x1);
                    fh[d] = pack_bf16x2(x0 * cs - x1 * sn, x0 * sn + x1 * cs);
                }
                *(u32x4 *)src = ft;
                *(u32x4 *)(sKh + gm_at<E, RK>(r, 8 * cc)) = fh;
            }
        };
#pragma unroll
        for (int i = 0; i < D - 1; ++i) issue(i);
        wait_next();
        transform(0);
        for (int i = 0; i < nb; ++i) {
            lds_only_barrier();                  // block i (its features formed) handed over
            issue(i + D - 1);                    // refills the slot of block i - 1
            if (i + 1 < nb) {
                wait_next();
                transform(i + 1);
            }
        }
        wait_vmcnt<0>();
        return;
    }
    if (w >= NCOMP) {
        // ---------------- loader waves ----------------
        // loaders 0, 1: halves of the key copies (0 also the betas); 2, 3:
        // halves of the value copies.  Rows past the split repeat its last
        // token (their beta is zeroed where it is used).  Every iteration
        // issues the same number of copies so that the waits below count
        // right: past the last block the last block is copied again, into the
        // slot of the missing block ii (the slot just released, which no
        // compute wave reads again).
        const int ld = w - NCOMP;
        const bool keys = ld < 2;
        auto issue = [&](int ii) {
            const int i = min(ii, nb - 1);
            const int t0 = t_lo + 64 * i, rmax = t_hi - 1 - t0;
            const size_t row0 = (row_b + t0) * p.H + h;
            unsigned char *sl = slot(ii);
#define GDN_SUM_DST(off) ((__attribute__((address_space(3))) void *)(sl + (off)))
            if (keys) {
                const char *base = (const char *)(p.k + row0 * DK);
                const unsigned rstride = (unsigned)(p.H * DK * ESZ);
#pragma unroll
                for (int j = 0; j < NCK2; ++j) {
                    const int ci = (ld & 1) * NCK2 + j;
                    int r, c;
                    gm_src<RK>(ci, l, r, c);
                    __builtin_amdgcn_global_load_lds(
                        (const void *)(base + (unsigned)min(r, rmax) * rstride + 16u * (unsigned)c),
                        GDN_SUM_DST(L::oK + 1024 * ci), 16, 0, 0);
                }
                if (ld == 0) {
                    const char *bb = (const char *)(p.beta + row0);
                    __builtin_amdgcn_global_load_lds(
                        (const void *)(bb + (unsigned)min(l, rmax) * (unsigned)(4 * p.H)), GDN_SUM_DST(L::oB), 4, 0, 0);
                }
            } else {
                const char *base = (const char *)(p.v + row0 * DV);
                const unsigned rstride = (unsigned)(p.H * DV * ESZ);
#pragma unroll
                for (int j = 0; j < NCV2; ++j) {
                    const int ci = (ld & 1) * NCV2 + j;
                    int r, c;
                    gm_src<RV>(ci, l, r, c);
                    __builtin_amdgcn_global_load_lds(
                        (const void *)(base + (unsigned)min(r, rmax) * rstride + 16u * (unsigned)c),
                        GDN_SUM_DST(L::oV + 1024 * ci), 16, 0, 0);
                }
            }
#undef GDN_SUM_DST
        };
        // block i has landed once at most D - 2 younger blocks are in flight
        auto wait_oldest = [&]() {
            if (ld == 0) wait_vmcnt<(D - 2) * (NCK2 + 1)>();
            else if (ld == 1) wait_vmcnt<(D - 2) * NCK2>();
            else wait_vmcnt<(D - 2) * NCV2>();
        };
#pragma unroll
        for (int i = 0; i < D - 1; ++i) issue(i);
        for (int i = 0; i < nb; ++i) {
            wait_oldest();
            lds_only_barrier();                  // block i handed to the compute waves
            issue(i + D - 1);                    // refills the slot of block i - 1
        }
        wait_vmcnt<0>();
        return;
    }

    // ---------------- compute waves ----------------
    const bool gw = w < 4;                                            // G waves (4..7: A waves)
    const bool zgw = FUSED && w >= 8;                                 // unrotated Gram waves (FUSED)
    const int wq = w & 3, kbw = wq % NP, c0 = wq / NP;                // row pair, column share
    constexpr int CPW = CPG > CPA ? CPG : CPA;
    f32x4 acc[2][CPW];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int j = 0; j < CPW; ++j) acc[a][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    // normalizer: the A waves (FUSED: the unrotated Gram waves) of the first
    // column share also accumulate K^T B 1 (a column of ones as the value)
    // for their row pair
    f32x4 accz[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
    const bool zw = NORM && (FUSED ? zgw : (!gw && w < 8)) && c0 == 0;
    const frag ones = ones_frag<E>();

    // the block loop, specialised for G waves (GB) and A waves, so that it has
    // no branch inside: all operand reads of a block (the K^T fragments
    // multiplied by beta) are issued before its products, which start as the
    // reads return.  Nothing reads a slot after the barrier that hands the
    // next block over (the loaders then refill it).
    // role 0: G waves, 1: A waves, 2: unrotated Gram waves (FUSED)
    auto run = [&](auto role) {
        constexpr int RO = decltype(role)::value;
        constexpr bool GB = RO != 1;
        constexpr int NC = GB ? CPG : CPA;
        constexpr size_t oKey = (FUSED && RO != 2) ? L::oKh : L::oK;
        struct Ops {
            frag a[2], b[NC];
        };
        // the K^T fragments of k block kb of block i, multiplied by beta
        auto read_a = [&](int i, int kb, frag (&fa)[2]) {
            const unsigned char *sl = slot(i);
            const E *sK = (const E *)(sl + oKey);
            const float *sB = (const float *)(sl + L::oB);
            // betas of this lane's 8 k-slots: tokens 32 kb + 8 lg + q'
            const f32x4 be0 = *(const f32x4 *)(sB + 32 * kb + 8 * lg);
            const f32x4 be1 = *(const f32x4 *)(sB + 32 * kb + 8 * lg + 4);
#pragma unroll
            for (int a = 0; a < 2; ++a) fa[a] = tr_frag_gm<E, RK>(sK, 32 * kb, 32 * kbw, true, a, li, lg);
            const int nvalid = t_hi - (t_lo + 64 * i + 32 * kb + 8 * lg);
            float bt[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) bt[q] = q < nvalid ? (q < 4 ? be0[q] : be1[q - 4]) : 0.f;
#pragma unroll
            for (int a = 0; a < 2; ++a) fa[a] = scale_frag(fa[a], bt);
        };
        // the B fragments of column tiles J0 .. J0 + NB - 1 of the wave's share
        auto read_b = [&](int i, int kb, int J0, auto nb_, frag *fb) {
            constexpr int NB = decltype(nb_)::value;
            const unsigned char *sl = slot(i);
            const E *sK = (const E *)(sl + oKey), *sV = (const E *)(sl + L::oV);
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const int c = c0 * NC + J0 + j;
                if constexpr (GB)
                    fb[j] = tr_frag_gm<E, RK>(sK, 32 * kb, 32 * (c >> 1), true, c & 1, li, lg);
                else
                    fb[j] = tr_frag_gm<E, RV>(sV, 32 * kb, 16 * c, false, 0, li, lg);
            }
        };
        auto read = [&](int i, int kb, Ops &o) {
            read_a(i, kb, o.a);
            read_b(i, kb, 0, std::integral_constant<int, NC>{}, o.b);
        };
        auto mul = [&](const Ops &o) {
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int j = 0; j < NC; ++j) acc[a][j] = TR::mma(o.a[a], o.b[j], acc[a][j]);
            if constexpr (NORM && (FUSED ? RO == 2 : RO == 1)) {
                if (zw) {
#pragma unroll
                    for (int a = 0; a < 2; ++a) accz[a] = TR::mma(o.a[a], ones, accz[a]);
                }
            }
        };
        Ops o0, o1;
        // split partials keep a Gram matrix's tiles on and above the diagonal
        // only: a Gram wave whose first half of column tiles lies wholly below
        // its row pair skips it
        const bool skip0 = FUSED && GB && p.NS > 1 && c0 * NC + NC / 2 <= 2 * kbw;
        for (int i = 0; i < nb; ++i) {
            // the barrier also completes the previous block's reads, so the
            // loaders may refill that block's slot
            lds_only_barrier();                  // block i has landed (FUSED: its features formed)
            if constexpr (FUSED) {
                // 16 waves leave 128 registers each: per k block the K^T
                // fragments, then the B fragments half the column tiles at a
                // time, each half multiplied as it arrives
                constexpr int NH = NC / 2;
                static_assert(NC % 2 == 0, "two halves of the column tiles");
#pragma unroll
                for (int kb = 0; kb < 2; ++kb) {
                    frag fa[2], fb[NH];
#pragma unroll
                    for (int hf = 0; hf < 2; ++hf) {
                        if (hf == 0 && skip0) continue;
                        if (hf == 0 || skip0) read_a(i, kb, fa);
                        read_b(i, kb, hf * NH, std::integral_constant<int, NH>{}, fb);
#pragma unroll
                        for (int a = 0; a < 2; ++a)
#pragma unroll
                            for (int j = 0; j < NH; ++j)
                                acc[a][hf * NH + j] = TR::mma(fa[a], fb[j], acc[a][hf * NH + j]);
                    }
                    if constexpr (NORM && RO == 2) {
                        if (zw) {
#pragma unroll
                            for (int a = 0; a < 2; ++a) accz[a] = TR::mma(fa[a], ones, accz[a]);
                        }
                    }
                }
            } else {
                read(i, 0, o0);
                read(i, 1, o1);
                mul(o0);
                mul(o1);
            }
        }
    };
    if (gw)
        run(std::integral_constant<int, 0>{});
    else if (zgw)
        run(std::integral_constant<int, 2>{});
    else
        run(std::integral_constant<int, 1>{});

    const size_t fi = (size_t)bh * p.F + f;
    const bool gram = gw || zgw;
    const int cpw = gram ? CPG : CPA;
    if (p.NS == 1) {
        const float ks = p.key_scale;
        if (gram) {
            const float k2 = ks * ks;
            E *dstg = zgw ? p.Gzf : p.Gf;
#pragma unroll
            for (int j = 0; j < CPG; ++j) {
                const int t = c0 * CPG + j;                             // G column tile (P32)
                TR::store8(dstg + ((fi * NR + t) * KBN + kbw) * 512 + l * 8,
                           TR::cat(TR::from_f32(acc[0][j] * k2), TR::from_f32(acc[1][j] * k2)));
            }
            if (FUSED && zw) {
#pragma unroll
                for (int a = 0; a < 2; ++a)
                    *(f32x4 *)(p.Af + ((fi * NR + 2 * kbw + a) * NJA + NCA) * 256 + l * 4) = accz[a] * ks;
            }
        } else {
            if (p.sum_mode != 2) {
#pragma unroll
                for (int j = 0; j < CPA; ++j) {
                    const int jt = c0 * CPA + j;
#pragma unroll
                    for (int a = 0; a < 2; ++a)
                        *(f32x4 *)(p.Af + ((fi * NR + 2 * kbw + a) * NJA + jt) * 256 + l * 4) = acc[a][j] * ks;
                }
            }
            if (!FUSED && zw && p.sum_mode != 1) {
#pragma unroll
                for (int a = 0; a < 2; ++a)
                    *(f32x4 *)(p.Af + ((fi * NR + 2 * kbw + a) * NJA + NCA) * 256 + l * 4) = accz[a] * ks;
            }
        }
    } else {
        // the Gram matrices are symmetric: only the tiles on and above the
        // diagonal (column tile >= row tile) go to the partials
        const int NC = gram ? NCG : NJA;
        float *dst = (gw ? p.PG : zgw ? p.PGz : p.PA) + (fi * p.NS + s) * (size_t)NR * NC * 256;
        if (gram || p.sum_mode != 2) {
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int j = 0; j < CPW; ++j)
                    if (j < cpw && (!gram || c0 * cpw + j >= 2 * kbw + a))
                        *(f32x4 *)(dst + ((size_t)((2 * kbw + a) * NC + c0 * cpw + j) * 64 + l) * 4) = acc[a][j];
        }
        if (zw && (FUSED || p.sum_mode != 1)) {
            // the A partials' normalizer tile (FUSED: written by the unrotated Gram waves)
            float *dz = p.PA + (fi * p.NS + s) * (size_t)NR * NJA * 256;
#pragma unroll
            for (int a = 0; a < 2; ++a)
                *(f32x4 *)(dz + ((size_t)((2 * kbw + a) * NJA + NCA) * 64 + l) * 4) = accz[a];
        }
    }
}

// Sum over the splits.  Items per (frame, head): the Dk/16 x Dk/32 G operand
// fragments, then the Dk/16 x Dv/16 A tiles, then (FUSED) the unrotated-key G
// fragments; one wave per item.  The splits store a Gram matrix's tiles on and
// above the diagonal only; a tile below it is its mirror's sum transposed
// through LDS: lane (li, lg) value q of tile (r, c) is lane
// (4 lg + q) + 16 (li / 4) value li % 4 of tile (c, r) (both P32 ordered).
template <class E, int DK, int DV, bool NORM, bool FUSED = false>
__global__ __launch_bounds__(256) void gdn_frame_reduce_kernel(FrameParams<E> p) {
    using TR = Tr<E>;
    constexpr int NR = DK / 16, KB = DK / 32, NCV = DV / 16 + NORM;
    constexpr int NGI = NR * KB, NAI = NR * NCV, NI = NGI + NAI + (FUSED ? NGI : 0);
    const int item = blockIdx.y * 4 + (threadIdx.x >> 6);
    const size_t fi = blockIdx.x;                                // (b*H + h) * F + f
    if (item >= NI) return;
    const int l = threadIdx.x & 63, li = l & 15, lg = l >> 4;
    const bool gz = FUSED && item >= NGI + NAI;
    // the sum over the splits of the f32x4 at src + s * stride, in split
    // order, four loads in flight at a time
    auto split_sum = [&](const float *src, size_t stride) {
        f32x4 x = {0.f, 0.f, 0.f, 0.f};
        int s = 0;
        for (; s + 4 <= p.NS; s += 4) {
            const f32x4 a0 = *(const f32x4 *)(src + (size_t)s * stride);
            const f32x4 a1 = *(const f32x4 *)(src + (size_t)(s + 1) * stride);
            const f32x4 a2 = *(const f32x4 *)(src + (size_t)(s + 2) * stride);
            const f32x4 a3 = *(const f32x4 *)(src + (size_t)(s + 3) * stride);
            x += a0;
            x += a1;
            x += a2;
            x += a3;
        }
        for (; s < p.NS; ++s) x += *(const f32x4 *)(src + (size_t)s * stride);
        return x;
    };
    if (item < NGI || gz) {
        __shared__ float tsm[4][256];                            // one transposition tile per wave
        float *ts = tsm[threadIdx.x >> 6];
        const int gi = gz ? item - NGI - NAI : item;
        const int t = gi / KB, kb = gi - t * KB;
        const float *src = (gz ? p.PGz : p.PG) + fi * p.NS * (size_t)NR * NR * 256 + l * 4;
        // tile (r, t) of the sum: stored if t >= r, else the mirror (t, r) transposed
        auto tile = [&](int r) {
            const bool up = t >= r;
            const size_t off = (size_t)(up ? r * NR + t : t * NR + r) * 256;
            const f32x4 x = split_sum(src + off, (size_t)NR * NR * 256);
            if (up) return x;
            *(f32x4 *)(ts + 4 * l) = x;
            f32x4 y;
#pragma unroll
            for (int q = 0; q < 4; ++q) y[q] = ts[4 * ((4 * lg + q) + 16 * (li >> 2)) + (li & 3)];
            return y;
        };
        const f32x4 lo = tile(2 * kb), hi = tile(2 * kb + 1);
        const float k2 = p.key_scale * p.key_scale;
        TR::store8((gz ? p.Gzf : p.Gf) + ((fi * NR + t) * KB + kb) * 512 + l * 8,
                   TR::cat(TR::from_f32(lo * k2), TR::from_f32(hi * k2)));
    } else {
        const int a = item - NGI;                                // = t * NCV + jt
        const float *src = p.PA + fi * p.NS * (size_t)NR * NCV * 256 + (size_t)a * 256 + l * 4;
        const f32x4 sum = split_sum(src, (size_t)NR * NCV * 256);
        *(f32x4 *)(p.Af + (fi * NR * NCV + a) * 256 + l * 4) = sum * p.key_scale;
    }
}

// Phase B.  One wave per (head, column tile jt): Hacc[t][q] =
// H[32 (t / 2) + 8 lg + 4 (t % 2) + q][16 jt + li], carried through the frames
// in fp32.  The product G H takes H rounded to E as the B operand.  A frame's
// G fragments and A tiles do not depend on the state, so the next frame's are
// requested before the current frame is computed (two register sets, used
// alternately; bf16 only, the fp32 fragments are twice as large).
// BIDIR (the bidirectional form, Algorithm Phase B): the wave first sweeps
// the frames F-1 .. 1 from a zero state, each frame's update applied to the
// later frames' history, and keeps the history Hb_f of every frame (zero for
// the last) in fp32 in Hb, lane by lane in the accumulator layout; the
// forward sweep then reads Hb_f with frame f's operands and writes
// H_f + Hb_f, rounded once, as the output operand.  The terminal state is the
// forward one.  FUSED: the normalizer tile takes the unrotated-key Gram
// matrix (the other tiles the rotated one).
template <class E> struct FrameScanPrefetch { static constexpr bool value = sizeof(E) == 2; };

template <class E, int DK, int DV, bool NORM, bool BIDIR, bool FUSED = false>
__global__ __launch_bounds__(64) void gdn_frame_scan_kernel(FrameParams<E> p) {
    using TR = Tr<E>;
    using frag = typename TR::frag;
    constexpr int NT = DK / 16, KB = DK / 32, NJ = DV / 16 + NORM;    // NORM: tile DV / 16 carries z
    int bh, jt;
    xcd_unit(blockIdx.x, NJ, bh, jt);
    if (bh >= p.B * p.H) return;
    const int b = bh / p.H, h = bh - b * p.H;
    const int l = threadIdx.x & 63, li = l & 15, lg = l >> 4;
    const int col = 16 * jt + li;
    const bool ztile = NORM && jt == DV / 16;                         // every column of this tile is z
    f32x4 Hacc[NT];
    // this wave's history tiles of frame f (BIDIR)
    auto hist = [&](int f) { return p.Hb + (((size_t)bh * p.F + f) * NJ + jt) * (size_t)NT * 256 + l * 4; };
    // a frame's operands: G fragments, A tiles, the decay and, in the forward
    // sweep of BIDIR, the frame's backward history (one load group, so that
    // waiting for it never waits for a younger frame's loads)
    struct Ops {
        frag g[NT][KB];
        f32x4 av[NT], hb[NT];
        float a;
    };
    auto load_ops = [&](int f, Ops &o, auto with_hist) {
        const size_t fi = (size_t)bh * p.F + f;
        // FUSED: the normalizer follows the Gram matrix of the unrotated keys
        const E *G = ((FUSED && ztile) ? p.Gzf : p.Gf) + fi * NT * KB * 512 + l * 8;
        const float *A = p.Af + fi * NT * NJ * 256 + l * 4;
        o.a = p.alpha[((size_t)b * p.F + f) * p.H + h];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) o.g[t][kb] = TR::load8(G + (t * KB + kb) * 512);
            o.av[t] = *(const f32x4 *)(A + (t * NJ + jt) * 256);
        }
        if constexpr (decltype(with_hist)::value) {
            const float *hp = hist(f);
#pragma unroll
            for (int t = 0; t < NT; ++t) o.hb[t] = *(const f32x4 *)(hp + t * 256);
        }
    };
    auto update = [&](const Ops &o) {
        frag hb[KB];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) hb[kb] = TR::cat(TR::from_f32(Hacc[2 * kb]), TR::from_f32(Hacc[2 * kb + 1]));
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            f32x4 gh = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) gh = TR::mma(o.g[t][kb], hb[kb], gh);
            Hacc[t] = o.a * (Hacc[t] - gh) + o.av[t];
        }
    };
    auto store_hist = [&](int f) {
        float *hp = hist(f);
#pragma unroll
        for (int t = 0; t < NT; ++t) *(f32x4 *)(hp + t * 256) = Hacc[t];
    };
    auto store_hf = [&](int f, const Ops &o) {
        E *hf = p.Hf + (((size_t)bh * p.F + f) * NJ + jt) * (size_t)KB * 512 + l * 8;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            f32x4 x0 = Hacc[2 * kb], x1 = Hacc[2 * kb + 1];
            if constexpr (BIDIR) {
                x0 += o.hb[2 * kb];
                x1 += o.hb[2 * kb + 1];
            }
            TR::store8(hf + kb * 512, TR::cat(TR::from_f32(x0), TR::from_f32(x1)));
        }
    };
    // n frames fid(0), fid(1), ..: load, update, then done(i, ops of step i)
    auto sweep = [&](int n, auto fid, auto with_hist, auto done) {
        Ops o0;
        if constexpr (FrameScanPrefetch<E>::value) {
            // the prefetch is unconditional (the last frame again past the
            // end) so the wait for a set always leaves exactly one younger set
            // in flight
            Ops o1;
            load_ops(fid(0), o0, with_hist);
            for (int i = 0; i < n; i += 2) {
                load_ops(fid(min(i + 1, n - 1)), o1, with_hist);
                update(o0);
                done(i, o0);
                if (i + 1 >= n) break;
                load_ops(fid(min(i + 2, n - 1)), o0, with_hist);
                update(o1);
                done(i + 1, o1);
            }
        } else {
            for (int i = 0; i < n; ++i) {
                load_ops(fid(i), o0, with_hist);
                update(o0);
                done(i, o0);
            }
        }
    };
    const int F = p.F;
    if constexpr (BIDIR) {
#pragma unroll
        for (int t = 0; t < NT; ++t) Hacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
        store_hist(F - 1);
        // step i applies frame F-1-i and gives the history of frame F-2-i
        if (F > 1)
            sweep(F - 1, [&](int i) { return F - 1 - i; }, std::false_type{},
                  [&](int i, const Ops &) { store_hist(F - 2 - i); });
        wait_vmcnt<0>();                         // the histories are written before they are read
    }
    if (ztile) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int r0 = 32 * (t >> 1) + 8 * lg + 4 * (t & 1);
#pragma unroll
            for (int q = 0; q < 4; ++q)
                Hacc[t][q] = p.z_in ? p.z_in[(size_t)bh * DK + r0 + q] : 0.f;
        }
    } else if (p.state_in) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int r0 = 32 * (t >> 1) + 8 * lg + 4 * (t & 1);
#pragma unroll
            for (int q = 0; q < 4; ++q) Hacc[t][q] = p.state_in[((size_t)bh * DK + r0 + q) * DV + col];
        }
    } else {
#pragma unroll
        for (int t = 0; t < NT; ++t) Hacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    sweep(F, [](int i) { return i; }, std::integral_constant<bool, BIDIR>{},
          [&](int i, const Ops &o) { store_hf(i, o); });
    if (ztile) {
        if (p.z_out && li == 0) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int r0 = 32 * (t >> 1) + 8 * lg + 4 * (t & 1);
#pragma unroll
                for (int q = 0; q < 4; ++q) p.z_out[(size_t)bh * DK + r0 + q] = Hacc[t][q];
            }
        }
    } else if (p.state_out) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int r0 = 32 * (t >> 1) + 8 * lg + 4 * (t & 1);
#pragma unroll
            for (int q = 0; q < 4; ++q) p.state_out[((size_t)bh * DK + r0 + q) * DV + col] = Hacc[t][q];
        }
    }
}

// Phase C.  Workgroup blk of a (frame, head) unit takes the 16-token tiles
// [TPW blk, TPW (blk + 1)) of the frame, wave w every WAVES-th of them from w.
// H_f's fragments are staged in LDS once per workgroup: lane (li, lg) of
// fragment (jo, kb) holds H_f[32 kb + 8 lg + q'][16 jo + li], the A operand of
// row 16 jo + li of H_f^T.  With the query rows as B operand the product tile
// is O^T, and lane (li, lg) gets O[token li][16 jo + 4 lg + q].  Each wave
// streams its tiles with the next tile's queries in flight.  The 16 x Dv
// result goes through LDS so that global stores write whole rows.
// NORM: every column of the extra column tile of H_f holds z, so every lane
// (li, lg) of its product holds the denominator z . q of token li; it is
// formed first and every output element is divided by it plus eps.
constexpr int kFrameOutWgs = 768;                  // output workgroups to aim for (3 per CU; swept)

// waves per output workgroup, one staging tile each (measured best: 4 for the
// numerator-only readout, 6 with the normalizer's extra product tile)
template <bool NORM> constexpr int frame_out_waves() { return NORM ? 6 : 4; }

template <class E, int DK, int DV, bool NORM> struct FrameOutLds {
    static constexpr int WAVES = frame_out_waves<NORM>();
    static constexpr int NJ = DV / 16 + NORM;
    static constexpr int LDO = DV + 16 / (int)sizeof(E);       // staged output row stride
    static constexpr size_t oO = sizeof(E) * DK * 16 * NJ;     // after H_f: one 16-row tile per wave
    static constexpr size_t bytes = oO + sizeof(E) * WAVES * 16 * LDO;
};

template <class E, int DK, int DV, bool NORM>
__global__ __launch_bounds__(64 * frame_out_waves<NORM>()) void gdn_frame_output_kernel(FrameParams<E> p) {
    using TR = Tr<E>;
    using frag = typename TR::frag;
    using LO = FrameOutLds<E, DK, DV, NORM>;
    constexpr int KB = DK / 32, NV = DV / 16, NJ = LO::NJ;
    constexpr int HV = NJ * 16 * DK * (int)sizeof(E) / 16;    // 16-byte vectors of H_f
    extern __shared__ __align__(16) unsigned char smem[];
    int unit, blk;
    xcd_unit(blockIdx.x, p.OB, unit, blk);
    if (unit >= p.F * p.B * p.H) return;
    const int bh = unit / p.F, f = unit - bh * p.F;
    const int b = bh / p.H, h = bh - b * p.H;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lg = l >> 4;
    const size_t fi = (size_t)bh * p.F + f;

    // H_f into LDS, every load of a thread in flight at once
    {
        constexpr int NTH = 64 * LO::WAVES, HIT = (HV + NTH - 1) / NTH;
        const u32x4 *src = (const u32x4 *)(p.Hf + fi * (size_t)NJ * 16 * DK);
        u32x4 hv[HIT];
#pragma unroll
        for (int it = 0; it < HIT; ++it)
            if (HV % NTH == 0 || tid + NTH * it < HV) hv[it] = src[tid + NTH * it];
#pragma unroll
        for (int it = 0; it < HIT; ++it)
            if (HV % NTH == 0 || tid + NTH * it < HV) ((u32x4 *)smem)[tid + NTH * it] = hv[it];
    }

    const size_t T = (size_t)p.F * p.N;
    const int ntf = (p.N + 15) / 16;                           // tiles in the frame
    const int tile_lo = blk * p.OTPW, tile_hi = min(ntf, tile_lo + p.OTPW);
    const size_t row_f = (size_t)b * T + (size_t)f * p.N;     // token rows of this frame
    // query fragments of tile i; rows past the frame read its last token
    auto load_q = [&](int i, frag (&qf)[KB]) {
        const int n = min(16 * i + li, p.N - 1);
        const E *qrow = p.q + ((row_f + n) * p.H + h) * DK;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) qf[kb] = load_frag<E>(qrow + 32 * kb, lg);
    };
    const E *sH = (const E *)smem + l * 8;
    E *sO = (E *)(smem + LO::oO) + w * 16 * LO::LDO;
    constexpr int VE = 16 / (int)sizeof(E);                   // elements per 16-byte vector
    constexpr int RV = DV / VE;                                // vectors per output row
    auto tile_product = [&](int jo, const frag (&qf)[KB]) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) acc = TR::mma(TR::load8(sH + (jo * KB + kb) * 512), qf[kb], acc);
        return acc;
    };
    auto compute = [&](int tile, const frag (&qf)[KB]) {
        if constexpr (NORM) {
            // every numerator product first, then the denominator of token li:
            // no product waits for the division
            f32x4 acc[NV];
#pragma unroll
            for (int jo = 0; jo < NV; ++jo) acc[jo] = tile_product(jo, qf);
            const float inv = 1.f / (tile_product(NV, qf)[0] + p.eps);
#pragma unroll
            for (int jo = 0; jo < NV; ++jo)
                TR::store(sO + li * LO::LDO + 16 * jo + 4 * lg, TR::from_f32(acc[jo] * inv));
        } else {
#pragma unroll
            for (int jo = 0; jo < NV; ++jo)
                TR::store(sO + li * LO::LDO + 16 * jo + 4 * lg, TR::from_f32(tile_product(jo, qf)));
        }
        // rows r of the tile, RV lanes per row, 64 / RV rows per pass
#pragma unroll
        for (int pass = 0; pass < 16 * RV / 64; ++pass) {
            const int r = pass * (64 / RV) + l / RV, c = (l % RV) * VE;
            const u32x4 val = *(const u32x4 *)(sO + r * LO::LDO + c);
            const int n = 16 * tile + r;
            if (tile < tile_hi && n < p.N) *(u32x4 *)(p.out + ((row_f + n) * p.H + h) * DV + c) = val;
        }
    };
    // the prefetch is unconditional (clamped to the workgroup's last tile) so
    // the wait for one buffer always leaves exactly the other in flight
    auto clampi = [&](int i) { return min(i, tile_hi - 1); };
    frag qa[KB], qb[KB];
    const int i0 = tile_lo + w;
    load_q(clampi(i0), qa);
    lds_barrier();
    constexpr int SW = LO::WAVES;
    for (int i = i0; i < tile_hi; i += 2 * SW) {
        load_q(clampi(i + SW), qb);
        compute(i, qa);
        if (i + SW >= tile_hi) break;
        load_q(clampi(i + 2 * SW), qa);
        compute(i + SW, qb);
    }
}

// Phase C of the fused operator (bf16).  As gdn_frame_output_kernel (each
// workgroup a run of 16-token tiles of one (frame, head), wave w every
// kFusedOutWaves-th tile from w, the next tile's loads in flight), with the
// query features formed on load and the gate and the per-head projection
// applied before the store.  Lane (li, lg) holds token li, channels
// 32 kb + 8 lg + q' of k block kb:
//   q~ = ReLU(gain_q o q / rms(q))   (the sum of squares reduced over the 4
//                                     lanes of the token),  q^ = R q~ (RoPE);
//   numerator tiles H_f^T q^, normalizer tile z . q~ (every column holds z);
//   y = SiLU(gate) o numerator / (z . q~ + eps);   out^T = W_o y^T.
// The value channels are dealt to the numerator tiles, and the output
// channels to the projection tiles, in the order of fused_out_chan: row
// 4 m + q of tile 2 kb + e is channel 32 kb + 8 m + 4 e + q.  Lane (li, lg)
// then holds channels 32 kb + 8 lg .. 32 kb + 8 lg + 7 of tiles 2 kb and
// 2 kb + 1, which are at once a 16-byte piece of the token's gate row, the
// projection's B operand fragment over k block kb (y never leaves the
// registers) and a 16-byte piece of its output row.  The H_f and W_o
// fragments take that order as they are staged into LDS.
constexpr int kFusedOutWaves = 12;

// Channel of row i (0 .. 15) of numerator or projection tile jo.
__device__ __forceinline__ int fused_out_chan(int jo, int i) {
    return 32 * (jo >> 1) + 8 * (i >> 2) + 4 * (jo & 1) + (i & 3);
}

template <int DK, int DV> struct FusedOutLds {
    static constexpr int NJ = DV / 16 + 1;
    static constexpr size_t oW = (size_t)2 * DK * 16 * NJ;      // after H_f: W_o fragments
    // gain_q[DK], then per channel pair the turns per unit of time, latent
    // row and latent column (the pair's frequency / 2 pi on its axis, zero on
    // the other two)
    static constexpr size_t oP = oW + (size_t)2 * DV * DV;
    static constexpr size_t bytes = oP + (size_t)4 * (DK + 3 * (DK / 2));
};

template <int DK, int DV>
__global__ __launch_bounds__(kFusedOutWaves * 64) void gdn_frame_output_fused_kernel(FrameParams<uint16_t> p) {
    using E = uint16_t;
    using TR = Tr<E>;
    using frag = TR::frag;
    using LO = FusedOutLds<DK, DV>;
    constexpr int KB = DK / 32, NV = DV / 16, NJ = LO::NJ, KBV = DV / 32;
    constexpr int NTH = kFusedOutWaves * 64;
    extern __shared__ __align__(16) unsigned char smem[];
    int unit, blk;
    xcd_unit(blockIdx.x, p.OB, unit, blk);
    if (unit >= p.F * p.B * p.H) return;
    const int bh = unit / p.F, f = unit - bh * p.F;
    const int b = bh / p.H, h = bh - b * p.H;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lg = l >> 4;
    const size_t fi = (size_t)bh * p.F + f;

    // H_f fragments (jo, kb): lane l holds row l % 16 of tile jo (channel
    // fused_out_chan(jo, l % 16); the normalizer tile as written) over
    // k slots 32 kb + 8 (l / 16) ..; W_o fragments (jo, kb): lane l holds
    // W_o[h][fused_out_chan(jo, l % 16)][32 kb + 8 (l / 16) ..]; the prologue
    // constants
    {
        constexpr int HV = NJ * 16 * DK * 2 / 16, HIT = (HV + NTH - 1) / NTH;
        constexpr int WV = DV * DV * 2 / 16, WIT = (WV + NTH - 1) / NTH;
        const u32x4 *src = (const u32x4 *)(p.Hf + fi * (size_t)NJ * 16 * DK);
        u32x4 hv[HIT], wv[WIT];
#pragma unroll
        for (int it = 0; it < HIT; ++it) {
            const int d = tid + NTH * it;
            if (HV % NTH == 0 || d < HV) {
                const int rec = d >> 6, ll = d & 63, jo = rec / KB, kb = rec - jo * KB;
                int sd = d;
                if (jo < NV) {
                    const int c = fused_out_chan(jo, ll & 15);
                    sd = (((c >> 4) * KB + kb) << 6) + (c & 15) + (ll & 48);
                }
                hv[it] = src[sd];
            }
        }
#pragma unroll
        for (int it = 0; it < WIT; ++it) {
            const int j = min(tid + NTH * it, WV - 1), fr = j >> 6, ll = j & 63, jo = fr / KBV, kb = fr - jo * KBV;
            wv[it] = *(const u32x4 *)(p.w_o + ((size_t)h * DV + fused_out_chan(jo, ll & 15)) * DV + 32 * kb +
                                      8 * (ll >> 4));
        }
        float *cp = (float *)(smem + LO::oP);
        for (int j = tid; j < DK + 3 * (DK / 2); j += NTH) {
            if (j < DK) {
                cp[j] = p.gain_q[h * DK + j];
            } else {
                const int pr = (j - DK) / 3, axis = (j - DK) - 3 * pr, a = p.rope_axis[pr];
                cp[j] = (a == axis || (axis == 2 && a != 0 && a != 1)) ? p.rope_freq[pr] * kInvTwoPi : 0.f;
            }
        }
#pragma unroll
        for (int it = 0; it < HIT; ++it)
            if (HV % NTH == 0 || tid + NTH * it < HV) ((u32x4 *)smem)[tid + NTH * it] = hv[it];
#pragma unroll
        for (int it = 0; it < WIT; ++it)
            if (WV % NTH == 0 || tid + NTH * it < WV) ((u32x4 *)(smem + LO::oW))[tid + NTH * it] = wv[it];
    }

    const size_t T = (size_t)p.F * p.N;
    const int ntf = (p.N + 15) / 16;
    const int tile_lo = blk * p.OTPW, tile_hi = min(ntf, tile_lo + p.OTPW);
    const size_t row_f = (size_t)b * T + (size_t)f * p.N;
    // query fragments and gate pieces (channels 32 kb + 8 lg ..) of tile i;
    // rows past the frame read its last token
    auto load = [&](int i, frag (&qf)[KB], u32x4 (&gt)[KBV]) {
        const int n = min(16 * i + li, p.N - 1);
        const size_t row = (row_f + n) * p.H + h;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) qf[kb] = load_frag<E>(p.q + row * DK + 32 * kb, lg);
#pragma unroll
        for (int kb = 0; kb < KBV; ++kb) gt[kb] = *(const u32x4 *)(p.gate + row * DV + 32 * kb + 8 * lg);
    };
    const E *sH = (const E *)smem + l * 8;
    const E *sW = (const E *)(smem + LO::oW) + l * 8;
    const float *cgain = (const float *)(smem + LO::oP), *cang = cgain + DK;
    auto compute = [&](int tile, const frag (&qf)[KB], const u32x4 (&gt)[KBV]) {
        // an offset the compiler cannot see through, so that the H_f and W_o
        // fragments are read from LDS where they are used rather than held in
        // registers across the tile loop
        int lo = 0;
        asm volatile("" : "+v"(lo));
        const E *tH = sH + lo, *tW = sW + lo;
        // prologue: features of token li
        float x[KB][8];
        float ss = 0.f;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                x[kb][2 * d] = __uint_as_float(qf[kb][d] << 16);
                x[kb][2 * d + 1] = __uint_as_float(qf[kb][d] & 0xffff0000u);
                ss += x[kb][2 * d] * x[kb][2 * d] + x[kb][2 * d + 1] * x[kb][2 * d + 1];
            }
        ss += __shfl_xor(ss, 16);
        ss += __shfl_xor(ss, 32);
        const float inv = rsqrtf(ss * (1.f / DK) + p.rms_eps);
        // token li's time, latent row and latent column
        const int n = min(16 * tile + li, p.N - 1);
        const int yc = n / p.lat_w;
        const float ct = (float)(p.t0 + f), cy = (float)yc, cx = (float)(n - yc * p.lat_w);
        frag qt[KB], qh[KB];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            const int ch = 32 * kb + 8 * lg;
            float xt[8], xh[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) xt[q] = fmaxf(cgain[ch + q] * x[kb][q] * inv, 0.f);
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                const float *ang = cang + 3 * (ch / 2 + d);
                float rv = ang[0] * ct + ang[1] * cy + ang[2] * cx;
                rv -= rintf(rv);
                const float sn = __builtin_amdgcn_sinf(rv), cs = __builtin_amdgcn_cosf(rv);
                xh[2 * d] = xt[2 * d] * cs - xt[2 * d + 1] * sn;
                xh[2 * d + 1] = xt[2 * d] * sn + xt[2 * d + 1] * cs;
            }
            qt[kb] = frag{pack_bf16x2(xt[0], xt[1]), pack_bf16x2(xt[2], xt[3]), pack_bf16x2(xt[4], xt[5]),
                          pack_bf16x2(xt[6], xt[7])};
            qh[kb] = frag{pack_bf16x2(xh[0], xh[1]), pack_bf16x2(xh[2], xh[3]), pack_bf16x2(xh[4], xh[5]),
                          pack_bf16x2(xh[6], xh[7])};
        }
        // the denominator of token li (every column of the normalizer tile is z)
        f32x4 dz = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) dz = TR::mma(TR::load8(tH + (NV * KB + kb) * 512), qt[kb], dz);
        const float invd = 1.f / (dz[0] + p.eps);
        // gated, normalized readout: numerator tiles 2 kb and 2 kb + 1 give
        // channels 32 kb + 8 lg .. + 7 of token li, the projection's B operand
        // over k block kb
        frag yb[KBV];
#pragma unroll
        for (int kv = 0; kv < KBV; ++kv) {
            float y[8];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kb = 0; kb < KB; ++kb)
                    acc = TR::mma(TR::load8(tH + ((2 * kv + e) * KB + kb) * 512), qh[kb], acc);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t gw = gt[kv][2 * e + (q >> 1)];
                    const float g = __uint_as_float((q & 1) ? (gw & 0xffff0000u) : (gw << 16));
                    y[4 * e + q] = g * __builtin_amdgcn_rcpf(1.f + __expf(-g)) * (acc[q] * invd);
                }
            }
            yb[kv] = frag{pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]), pack_bf16x2(y[4], y[5]),
                          pack_bf16x2(y[6], y[7])};
        }
        // projection: out^T = W_o y^T; tiles 2 kv and 2 kv + 1 give output
        // channels 32 kv + 8 lg .. + 7 of token li, stored as one 16-byte piece
        const bool live = tile < tile_hi && 16 * tile + li < p.N;
        E *orow = p.out + ((row_f + 16 * tile + li) * p.H + h) * DV + 8 * lg;
#pragma unroll
        for (int kv = 0; kv < KBV; ++kv) {
            f32x4 o[2];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                o[e] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kb = 0; kb < KBV; ++kb)
                    o[e] = TR::mma(TR::load8(tW + ((2 * kv + e) * KBV + kb) * 512), yb[kb], o[e]);
            }
            const u32x4 val = {pack_bf16x2(o[0][0], o[0][1]), pack_bf16x2(o[0][2], o[0][3]),
                               pack_bf16x2(o[1][0], o[1][1]), pack_bf16x2(o[1][2], o[1][3])};
            if (live) *(u32x4 *)(orow + 32 * kv) = val;
        }
    };
    // the prefetch is unconditional (clamped to the workgroup's last tile) so
    // the wait for one buffer always leaves exactly the other in flight
    constexpr int SW = kFusedOutWaves;
    auto clampi = [&](int i) { return min(i, tile_hi - 1); };
    frag qa[KB], qb[KB];
    u32x4 ga[KBV], gb[KBV];
    const int i0 = tile_lo + w;
    load(clampi(i0), qa, ga);
    lds_barrier();                                // staging complete
    for (int i = i0; i < tile_hi; i += 2 * SW) {
        load(clampi(i + SW), qb, gb);
        compute(i, qa, ga);
        if (i + SW >= tile_hi) break;
        load(clampi(i + 2 * SW), qa, ga);
        compute(i + SW, qb, gb);
    }
}

// ---------------------------------------------------------------------------
// The fused operator in fp32 (the paper's "ieee" precision mode, appendix "GDN
// Kernel Details", "Precision modes"): every feature, product and readout in
// fp32.  Phase A's feature maps are formed once per token by
// gdn_frame_features_kernel into the workspace; the summaries then run as the
// plain frame-wise summary kernel twice (rotated keys: G and A; unrotated
// keys: the normalizer's Gram matrix and K~^T beta); the split reduction and
// the scan are the fused variants; Phase C is gdn_frame_output_f32_fused_kernel
// (numerator on q^, normalizer on q~, gate) and gdn_frame_project_f32_kernel
// (the per-head projection).
// ---------------------------------------------------------------------------

// Features of every token row of q_raw and k_raw: with r(x) = gain o x /
// sqrt(mean_i x_i^2 + rms_eps),
//   q~ = ReLU(r_q(q)),  q^ = R q~,  k~ = feat_scale ReLU(r_k(k)),  k^ = R k~,
// R rotating channel pair (2i, 2i + 1) by rope_freq[i] times the token's
// coordinate on rope_axis[i] (0 time t0 + f, 1 latent row s / lat_w, else
// latent column s % lat_w).  One lane per channel pair, Dk / 2 lanes per row
// (the row's sum of squares reduced across them); the angle in fp64 and its
// sine and cosine by the accurate fp64 routine, so that long time coordinates
// cost no precision.
template <int DK>
__global__ __launch_bounds__(256) void gdn_frame_features_kernel(FrameParams<float> p) {
    constexpr int P = DK / 2;                                   // lanes per row
    const size_t nrow = (size_t)p.B * p.F * p.N * p.H;           // rows per tensor
    const int l = threadIdx.x & 63;
    const size_t r = ((size_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * (64 / P) + l / P;
    if (r >= 2 * nrow) return;
    const bool isk = r >= nrow;
    const size_t row = isk ? r - nrow : r;                       // (b T + t) H + h
    const int h = (int)(row % p.H);
    const int t = (int)((row / p.H) % ((size_t)p.F * p.N));
    const int f = t / p.N, sidx = t - f * p.N;
    const int i = l % P;
    const float2 x = *(const float2 *)((isk ? p.k : p.q) + row * DK + 2 * i);
    float ss = x.x * x.x + x.y * x.y;
#pragma unroll
    for (int o = P / 2; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
    const float inv = 1.f / sqrtf(ss * (1.f / DK) + p.rms_eps);
    const float *gain = (isk ? p.gain_k : p.gain_q) + (size_t)h * DK + 2 * i;
    const float sc = isk ? p.feat_scale : 1.f;
    const float x0 = sc * fmaxf(gain[0] * x.x * inv, 0.f), x1 = sc * fmaxf(gain[1] * x.y * inv, 0.f);
    const int ax = p.rope_axis[i];
    const int yc = sidx / p.lat_w;
    const double coord = ax == 0 ? (double)(p.t0 + f) : ax == 1 ? (double)yc : (double)(sidx - yc * p.lat_w);
    double sn, cs;
    sincos((double)p.rope_freq[i] * coord, &sn, &cs);
    const float s1 = (float)sn, c1 = (float)cs;
    float *ft = (isk ? p.fkt : p.fqt) + row * DK + 2 * i, *fh = (isk ? p.fkh : p.fqh) + row * DK + 2 * i;
    *(float2 *)ft = make_float2(x0, x1);
    *(float2 *)fh = make_float2(x0 * c1 - x1 * s1, x0 * s1 + x1 * c1);
}

// Phase C numerator, normalizer and gate in fp32: as gdn_frame_output_kernel
// with the normalizer (one 16-token tile per wave at a time, H_f of the
// (frame, head) in LDS), with the numerator tiles on q^, the normalizer tile
// on q~, and y = SiLU(gate) o numerator / (z . q~ + eps) written to ybuf.
template <int DK, int DV>
__global__ __launch_bounds__(64 * frame_out_waves<true>()) void gdn_frame_output_f32_fused_kernel(
    FrameParams<float> p) {
    using E = float;
    using TR = Tr<E>;
    using frag = typename TR::frag;
    using LO = FrameOutLds<E, DK, DV, true>;
    constexpr int KB = DK / 32, NV = DV / 16, NJ = LO::NJ;
    constexpr int HV = NJ * 16 * DK * (int)sizeof(E) / 16;    // 16-byte vectors of H_f
    extern __shared__ __align__(16) unsigned char smem[];
    int unit, blk;
    xcd_unit(blockIdx.x, p.OB, unit, blk);
    if (unit >= p.F * p.B * p.H) return;
    const int bh = unit / p.F, f = unit - bh * p.F;
    const int b = bh / p.H, h = bh - b * p.H;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lg = l >> 4;
    const size_t fi = (size_t)bh * p.F + f;
    {
        constexpr int NTH = 64 * LO::WAVES, HIT = (HV + NTH - 1) / NTH;
        const u32x4 *src = (const u32x4 *)(p.Hf + fi * (size_t)NJ * 16 * DK);
        u32x4 hv[HIT];
#pragma unroll
        for (int it = 0; it < HIT; ++it)
            if (HV % NTH == 0 || tid + NTH * it < HV) hv[it] = src[tid + NTH * it];
#pragma unroll
        for (int it = 0; it < HIT; ++it)
            if (HV % NTH == 0 || tid + NTH * it < HV) ((u32x4 *)smem)[tid + NTH * it] = hv[it];
    }
    const size_t T = (size_t)p.F * p.N;
    const int ntf = (p.N + 15) / 16;
    const int tile_lo = blk * p.OTPW, tile_hi = min(ntf, tile_lo + p.OTPW);
    const size_t row_f = (size_t)b * T + (size_t)f * p.N;
    // query features of tile i (rotated and unrotated); rows past the frame
    // read its last token
    auto load_q = [&](int i, frag (&qh)[KB], frag (&qt)[KB]) {
        const int n = min(16 * i + li, p.N - 1);
        const size_t o = ((row_f + n) * p.H + h) * DK;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            qh[kb] = load_frag<E>(p.fqh + o + 32 * kb, lg);
            qt[kb] = load_frag<E>(p.fqt + o + 32 * kb, lg);
        }
    };
    const E *sH = (const E *)smem + l * 8;
    E *sO = (E *)(smem + LO::oO) + w * 16 * LO::LDO;
    constexpr int RV = DV / 4;                                 // float4 per row
    auto tile_product = [&](int jo, const frag (&qf)[KB]) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) acc = TR::mma(TR::load8(sH + (jo * KB + kb) * 512), qf[kb], acc);
        return acc;
    };
    auto compute = [&](int tile, const frag (&qh)[KB], const frag (&qt)[KB]) {
        f32x4 acc[NV];
#pragma unroll
        for (int jo = 0; jo < NV; ++jo) acc[jo] = tile_product(jo, qh);
        const float inv = 1.f / (tile_product(NV, qt)[0] + p.eps);
        // lane (li, lg) holds columns 16 jo + 4 lg + q of token li
        const int n = min(16 * tile + li, p.N - 1);
        const float *grow = p.gate + ((row_f + n) * p.H + h) * DV;
#pragma unroll
        for (int jo = 0; jo < NV; ++jo) {
            const f32x4 g = *(const f32x4 *)(grow + 16 * jo + 4 * lg);
            f32x4 y;
#pragma unroll
            for (int q = 0; q < 4; ++q) y[q] = g[q] / (1.f + expf(-g[q])) * (acc[jo][q] * inv);
            *(f32x4 *)(sO + li * LO::LDO + 16 * jo + 4 * lg) = y;
        }
#pragma unroll
        for (int pass = 0; pass < 16 * RV / 64; ++pass) {
            const int r = pass * (64 / RV) + l / RV, c = (l % RV) * 4;
            const f32x4 val = *(const f32x4 *)(sO + r * LO::LDO + c);
            const int nn = 16 * tile + r;
            if (tile < tile_hi && nn < p.N) *(f32x4 *)(p.ybuf + ((row_f + nn) * p.H + h) * DV + c) = val;
        }
    };
    auto clampi = [&](int i) { return min(i, tile_hi - 1); };
    frag ha[KB], ta[KB], hb[KB], tb[KB];
    const int i0 = tile_lo + w;
    load_q(clampi(i0), ha, ta);
    lds_barrier();
    constexpr int SW = LO::WAVES;
    for (int i = i0; i < tile_hi; i += 2 * SW) {
        load_q(clampi(i + SW), hb, tb);
        compute(i, ha, ta);
        if (i + SW >= tile_hi) break;
        load_q(clampi(i + 2 * SW), ha, ta);
        compute(i + SW, hb, tb);
    }
}

// The per-head projection in fp32: out_n = W_o[h] ybuf_n.  Workgroup (run of 64
// tokens, b h): W_o[h] and the run's rows of ybuf staged in LDS with row
// stride DV + 4 (the 16 rows x 4 k slots an operand read touches fall in 64
// distinct banks); wave w takes tokens 16 w .. 16 w + 15 of the run and every
// 16-channel output tile on 16x16x4 fp32 MFMA, lane (li, lg) supplying
// W_o[16 it + li][4 kk + lg] and ybuf[token li][4 kk + lg]; the accumulator
// lane (li, lg) then holds channels 16 it + 4 lg .. + 3 of token li.
template <int DV> struct ProjectLds {
    static constexpr int LD = DV + 4;
    static constexpr size_t bytes = (size_t)4 * (DV + 64) * LD;
};

template <int DV>
__global__ __launch_bounds__(256) void gdn_frame_project_f32_kernel(FrameParams<float> p) {
    constexpr int LD = ProjectLds<DV>::LD, RV = DV / 4;
    extern __shared__ __align__(16) unsigned char smem[];
    float *sW = (float *)smem, *sY = sW + DV * LD;
    const size_t T = (size_t)p.F * p.N;
    const int bh = blockIdx.y, b = bh / p.H, h = bh - b * p.H;
    const int t0 = blockIdx.x * 64;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lg = l >> 4;
    for (int idx = tid; idx < DV * RV; idx += 256) {
        const int r = idx / RV, c = idx - r * RV;
        *(f32x4 *)(sW + r * LD + 4 * c) = *(const f32x4 *)(p.w_o + ((size_t)h * DV + r) * DV + 4 * c);
    }
    for (int idx = tid; idx < 64 * RV; idx += 256) {
        const int r = idx / RV, c = idx - r * RV;
        const size_t t = min((size_t)(t0 + r), T - 1);
        *(f32x4 *)(sY + r * LD + 4 * c) = *(const f32x4 *)(p.ybuf + (((size_t)b * T + t) * p.H + h) * DV + 4 * c);
    }
    __syncthreads();
    const float *yl = sY + (16 * w + li) * LD + lg;
    const size_t tok = (size_t)t0 + 16 * w + li;
#pragma unroll 2
    for (int it = 0; it < DV / 16; ++it) {
        const float *wl = sW + (16 * it + li) * LD + lg;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < DV / 4; ++kk) acc = mma_f32_k4(wl[4 * kk], yl[4 * kk], acc);
        if (tok < T) *(f32x4 *)(p.out + (((size_t)b * T + tok) * p.H + h) * DV + 16 * it + 4 * lg) = acc;
    }
}

}  // namespace gdn
