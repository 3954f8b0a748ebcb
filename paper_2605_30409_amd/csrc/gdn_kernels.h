// The gfx950 kernels of the GDN chunk forward.
//
// Notation (per batch b, head h; state H = S^T of shape [Dk][Dv]).  Inside a
// chunk of C = 64 tokens r = 0..63 with entry state H_0:
//   g_r   = sum_{s <= r} log alpha_s                    (log-space decay)
//   A     = strict_lower( beta_r e^{g_r - g_s} k_r . k_s )
//   T     = (I + A)^{-1}                                 (unit lower triangular)
//   W     = T diag(beta e^g) K,   Ut = T diag(beta) V    (WY factors)
//   U     = Ut - W H_0                                   (pseudo-values)
//   O     = diag(e^g) Q H_0 + (Q K^T o M) U,   M_rs = e^{g_r - g_s} (s <= r)
//   H_C   = e^{g_C} H_0 + (diag(e^{g_C - g}) K)^T U
// This is the recurrence S_t = alpha_t S_{t-1}(I - beta_t k_t k_t^T) +
// beta_t v_t k_t^T, o_t = S_t q_t, unrolled over the chunk: the token-wise
// analog of the paper's split into per-frame summaries and a short scan
// (Section "Efficient System Co-design", S_f = alpha_f P_f S_{f-1} + A_f; the
// three stages mirror its Phase A / B / C pipeline, appendix "GDN Kernel
// Details").  Decay ratios are formed as exp of log-space differences, with
// s > r masked before the exp.
//
// Workspace per (b*H + h, chunk) -- see gdn_api.hip for the byte layout:
//   g  [64]       fp64   cumulative log decay (fp64 so that g_r - g_s keeps
//                        its precision when the decay over a chunk is huge)
//   gf [68]       fp32   e^{g_C - g_r} (the update's per-token key scale),
//                        then g_C, the log decay over the chunk, as one fp64,
//                        and gamma = e^{g_C}
//   W  64*Dk      E      -W (the WY factor, negated), fragment-major for the scan
//   Ut Dv*64      E      Ut, fragment-major
//   Hs [Dv][Dk]   E      H_{c-1}^T, the state entering the chunk
//   Us [Dv][64]   E      U^T
// "Fragment-major" means the exact per-lane order in which the scan's MFMAs
// consume the operand, so every scan load is one contiguous wave access:
//   W  [Dk/64 wave][4 token tile][2 k block][64 lane][8]
//        = -W[32 m + p32_row(a, li)][64 wave + 32 kb + 8 lg + e]    (tile 2 m + a)
//   Ut [Dv/16 column tile][4 token tile][64 lane][4]
//        = Ut[32 m + 8 lg + 4 a + e][16 jt + li]                      (tile 2 m + a)
// The scan reads the keys from the input itself and applies their decay
// factors in registers: the update takes K^T (diag(e^{g_C - g}) U), so no
// scaled copy of K is written.
#pragma once

#include "gdn_device.h"

namespace gdn {

constexpr int kGateRec = kChunk + 4;  // floats per chunk gate record (see gf above)

template <class E> struct Params {
    const E *q, *k, *v;
    const float *alpha, *beta, *state_in;
    E *out;
    float *state_out;
    int B, H, T, NC;
    int G, NG;        // chunks per scan group, number of groups
    double *g;
    float *gf;        // per (b*H + h, chunk): e^{g_C - g_r} [64], g_C (fp64), e^{g_C}, 1 unused
    E *W, *Ut, *Hs, *Us;
    // Fused output (bf16, one scan group): the scan computes the output, from
    // Qf = diag(e^g) Q and Pf = (Q K^T o M) row fragments written by the WY
    // kernel (they reuse the Hs / Us workspace regions, which are then unused).
    int fused;
    E *Qf, *Pf;
    E *Nf;            // per (b*H + h, group): N_g = Phi_g - Gamma_g I, fragment-major
    float *PsiT;      // per (b*H + h, group): Psi_g^T [Dv][Dk]
    double *lgam;     // per (b*H + h, group): log Gamma_g
    float *HgT;       // per (b*H + h, group): entry state H^T [Dv][Dk]
};

// --------------------------------------------------------------------------
// Stage 1: per-chunk WY / UT transform.  Grid (NC, B*H), kWyWaves waves.
// --------------------------------------------------------------------------
// LDS: K rows, A (fp32; V rows take its place once the solve is done), T
// (fp32), gates.  52.3 KB on the bf16 path at D = 128: three workgroups per CU.
template <class E, int DK, int DV> struct WyLds {
    static constexpr int PAD = 16 / (int)sizeof(E);
    static constexpr int LDK = DK + PAD;      // K, row-major (token rows)
    static constexpr int LDV = DV + PAD;      // V, row-major
    static constexpr int LDA = kChunk + 4;    // A and T (fp32)
    static constexpr size_t szA = 4 * kChunk * LDA;
    static constexpr size_t szV = sizeof(E) * kChunk * LDV;
    static constexpr size_t oK = 0;
    static constexpr size_t oA = oK + sizeof(E) * kChunk * LDK;  // A, then V
    static constexpr size_t oT = oA + (szA > szV ? szA : szV);
    static constexpr size_t oG = oT + szA;
    static constexpr size_t bytes = oG + 8 * kChunk + 3 * 4 * kChunk;
    // waves per SIMD when as many eight-wave workgroups as fit in 160 KB share
    // a CU (the register budget the kernel is compiled for)
    static constexpr int fit = (int)((160 * 1024) / bytes);
    static constexpr int waves_per_simd = fit >= 4 ? 8 : (fit < 1 ? 2 : 2 * fit);
};

// Decay ratio e^{g_r - g_s} (s <= r) inside the WY kernel.  The fp32 path
// takes the difference of the fp64 cumulative sums (full precision even when
// the decay over a chunk is huge); the bf16 path takes it from fp32 copies of
// g * log2(e), whose rounding (at most ~1e-3 relative to the ratio when
// |g| ~ 5600, the extreme of a chunk of alpha ~ 0) is far below bf16's.
template <class E>
__device__ __forceinline__ float wy_decay(const double *sg, const float *sgl, int r, int s) {
    constexpr double kLog2e = 1.4426950408889634;
    if constexpr (sizeof(E) == 2)
        return __builtin_amdgcn_exp2f(sgl[r] - sgl[s]);
    else
        return __builtin_amdgcn_exp2f((float)((sg[r] - sg[s]) * kLog2e));
}

constexpr int kWyWaves = 8;

template <class E, int DK, int DV>
__global__ __launch_bounds__(64 * kWyWaves)
__attribute__((amdgpu_waves_per_eu(WyLds<E, DK, DV>::waves_per_simd))) void gdn_wy_kernel(Params<E> p) {
    using L = WyLds<E, DK, DV>;
    using TR = Tr<E>;
    using frag = typename TR::frag;
    constexpr int NWV = kWyWaves, NT = 64 * NWV;
    constexpr int VE = 16 / (int)sizeof(E);       // elements per 16-byte vector
    constexpr int NKV = kChunk * (DK / VE) / NT;   // K vectors per thread
    constexpr int NVV = kChunk * (DV / VE) / NT;   // V vectors per thread
    static_assert(NKV * NT == kChunk * (DK / VE) && NVV * NT == kChunk * (DV / VE), "whole vectors per thread");
    constexpr int NFR = (DK / 64) * 8;             // W fragments per chunk
    constexpr double kLog2e = 1.4426950408889634;
    extern __shared__ __align__(16) unsigned char smem[];
    E *sK = (E *)(smem + L::oK);
    float *sA = (float *)(smem + L::oA);
    E *sV = (E *)(smem + L::oA);                  // V rows, once A is dead
    float *sT = (float *)(smem + L::oT);
    double *sg = (double *)(smem + L::oG);        // g_r
    float *sb = (float *)(sg + kChunk);           // beta_r
    float *sw = sb + kChunk;                      // -beta_r e^{g_r}
    float *sgl = sw + kChunk;                     // g_r log2(e) in fp32 (bf16 path)

    const int c = blockIdx.x, bh = blockIdx.y;
    const int b = bh / p.H, h = bh - b * p.H;
    // w is wave-uniform: scalar branches and table lookups
    const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), l = tid & 63, li = l & 15,
              lg = l >> 4;
    const int t0 = c * kChunk;
    const int nvalid = min(kChunk, p.T - t0);
    const size_t cidx = (size_t)bh * p.NC + c;
    const size_t row0 = ((size_t)b * p.T + t0) * p.H + h;  // token-row index of token t0
    const size_t rstride = (size_t)p.H;                    // token-row stride

    // Gates first (they head the dependency chain), then K rows with 16-byte
    // coalesced loads (padding rows are zero).  The queries (first needed after
    // the A tiles) and V (needed only for U~ at the end) are requested after
    // the first barrier, so that the gate and K requests of all the workgroups
    // starting together are served first.
    float ga = 1.f, gbe = 0.f;  // alpha, beta of token l (wave 0; padding: 1, 0)
    if (w == 0 && l < nvalid) {
        ga = p.alpha[row0 + l * rstride];
        gbe = p.beta[row0 + l * rstride];
    }
    uint4 kreg[NKV], vreg[NVV];
#pragma unroll
    for (int n = 0; n < NKV; ++n) {
        const int idx = tid + NT * n, r = idx / (DK / VE), cv = idx % (DK / VE);
        kreg[n] = make_uint4(0u, 0u, 0u, 0u);
        if (r < nvalid) kreg[n] = *(const uint4 *)(p.k + (row0 + r * rstride) * DK + cv * VE);
    }
    // Fused output: six (token tile rt, s block m) jobs on waves 1..6, run
    // while wave 0 inverts the diagonal blocks: job j = w - 1 is (j, 0) for
    // j < 4 (these also write the tile's Qf) and (j - 2, 1) for j = 4, 5.
    // Q rows of the job's 16 tokens as row fragments (Q[r][32 kb + 8 lg + e],
    // r = 16 rt + li; padded tokens are 0).
    const int qj = w - 1;
    const int qjob_rt = qj < 4 ? qj : qj - 2, qjob_m = qj < 4 ? 0 : 1;
    const bool qjob = w >= 1 && w <= 6;
    const int rq = 16 * qjob_rt + li;
    frag qf[DK / 32];
    // Gates: wave-wide inclusive prefix sum of clamped log alpha in fp64
    // (padding tokens: alpha = 1, beta = 0).
    if (w == 0) {
        const float be = gbe;
        float la = logf(ga);
        la = (la < kLogAlphaMin) ? kLogAlphaMin : la;  // keeps NaN
        double g = (double)la;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const double o = __shfl_up(g, d);
            if (l >= d) g += o;
        }
        const double gC = __shfl(g, kChunk - 1);
        const float eg = __builtin_amdgcn_exp2f((float)(g * kLog2e));
        sg[l] = g;
        sgl[l] = (float)(g * kLog2e);
        sb[l] = be;
        sw[l] = -be * eg;
        p.g[cidx * kChunk + l] = g;
        p.gf[cidx * kGateRec + l] = __builtin_amdgcn_exp2f((float)((gC - g) * kLog2e));
        if (l == 0) {
            *(double *)(p.gf + cidx * kGateRec + kChunk) = gC;
            p.gf[cidx * kGateRec + kChunk + 2] = expf((float)gC);
        }
    }
#pragma unroll
    for (int n = 0; n < NKV; ++n) {
        const int idx = tid + NT * n, r = idx / (DK / VE), cv = idx % (DK / VE);
        *(uint4 *)(sK + r * L::LDK + cv * VE) = kreg[n];
    }
    lds_barrier();
    if constexpr (sizeof(E) == 2) {
        if (p.fused && qjob) {
#pragma unroll
            for (int kb = 0; kb < DK / 32; ++kb)
                qf[kb] = rq < nvalid ? load_frag<E>(p.q + (row0 + rq * rstride) * DK + 32 * kb, lg)
                                     : TR::cat(TR::zero(), TR::zero());
        }
    }
#pragma unroll
    for (int n = 0; n < NVV; ++n) {
        const int idx = tid + NT * n, r = idx / (DV / VE), cv = idx % (DV / VE);
        vreg[n] = make_uint4(0u, 0u, 0u, 0u);
        if (r < nvalid) vreg[n] = *(const uint4 *)(p.v + (row0 + r * rstride) * DV + cv * VE);
    }

    // A = strict_lower(beta_r e^{g_r - g_s} K K^T): the 10 lower 16x16 blocks.
    for (int t = w; t < 10; t += NWV) {
        const int bi = (t >= 6) ? 3 : (t >= 3) ? 2 : (t >= 1) ? 1 : 0;
        const int bj = t - bi * (bi + 1) / 2;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < DK / 32; ++kb)
            acc = TR::mma(load_frag<E>(sK + (16 * bi + li) * L::LDK + 32 * kb, lg),
                          load_frag<E>(sK + (16 * bj + li) * L::LDK + 32 * kb, lg), acc);
        const int s2 = 16 * bj + li;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int r = 16 * bi + 4 * lg + q;
            float val = 0.f;
            if (s2 < r) val = sb[r] * wy_decay<E>(sg, sgl, r, s2) * acc[q];
            sA[r * L::LDA + s2] = val;
        }
    }
    lds_barrier();

    // T = (I + A)^{-1} in fp32.  Wave 0 inverts the four diagonal 16x16 blocks
    // by forward substitution (lane = block * 16 + column) while waves 1..6
    // produce the fused-output score fragments, which need only Q, K and the
    // gates.
    if (w == 0) {
        const int base = 16 * (l >> 4), j = l & 15;
        float x[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float *arow = sA + (base + r) * L::LDA + base;
            float acc = (r == j) ? 1.f : 0.f;
#pragma unroll
            for (int s4 = 0; s4 < (r + 3) / 4; ++s4) {
                const f32x4 av = *(const f32x4 *)(arow + 4 * s4);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (4 * s4 + e < r) acc -= av[e] * x[4 * s4 + e];
            }
            x[r] = acc;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) sT[(base + r) * L::LDA + base + j] = x[r];
    } else {
        // Fused output: job (rt, m) writes, for token tile rt,
        //   Qf[rt][kb][lane][e] = e^{g_r} Q[r][32 kb + 8 lg + e]      (m = 0 jobs)
        //   Pf[rt][m][lane][e]  = e^{g_r - g_s} q_r . k_s (s <= r, else 0), s = 32 m + 8 lg + e,
        // the row fragments (B operands over d, resp. s) of the fused output.
        // P^T tiles take their s rows in P32 order, so a tile pair is one
        // fragment; block m = 1 only matters for r >= 32.
        if constexpr (sizeof(E) == 2) {
            if (p.fused && qjob) {
                if (qjob_m == 0) {
                    const float er = expf((float)sg[rq]);
                    E *Qf = p.Qf + cidx * (size_t)kChunk * DK + l * 8;
#pragma unroll
                    for (int kb = 0; kb < DK / 32; ++kb) {
                        const f32x4 lo = TR::to_f32(TR::lo(qf[kb])) * er, hi = TR::to_f32(TR::hi(qf[kb])) * er;
                        TR::store8(Qf + (size_t)(qjob_rt * (DK / 32) + kb) * 512,
                                   TR::cat(TR::from_f32(lo), TR::from_f32(hi)));
                    }
                }
                E *Pf = p.Pf + cidx * (size_t)kChunk * kChunk + l * 8;
                const int m = qjob_m;
                typename TR::quad pq[2];
#pragma unroll
                for (int a = 0; a < 2; ++a) {
                    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int kb = 0; kb < DK / 32; ++kb)
                        acc = TR::mma(load_frag<E>(sK + (32 * m + p32_row(a, li)) * L::LDK + 32 * kb, lg), qf[kb], acc);
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int s2 = 32 * m + 8 * lg + 4 * a + q;
                        acc[q] = (s2 <= rq) ? wy_decay<E>(sg, sgl, rq, s2) * acc[q] : 0.f;
                    }
                    pq[a] = TR::from_f32(acc);
                }
                TR::store8(Pf + (size_t)(qjob_rt * 2 + m) * 512, TR::cat(pq[0], pq[1]));
            }
        }
    }
    lds_barrier();
    // Off-diagonal blocks by block distance: T_ij = -T_ii sum_{m=j}^{i-1} A_im T_mj.
    for (int dist = 1; dist < 4; ++dist) {
        if (w < 4 - dist) {
            const int j = w, i = w + dist;
            f32x4 X = {0.f, 0.f, 0.f, 0.f};
            for (int m = j; m < i; ++m) {
                const f32x4 a = *(const f32x4 *)(sA + (16 * i + li) * L::LDA + 16 * m + 4 * lg);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    X = mma_f32_k4(a[q], sT[(16 * m + 4 * lg + q) * L::LDA + 16 * j + li], X);
            }
            const f32x4 a = *(const f32x4 *)(sT + (16 * i + li) * L::LDA + 16 * i + 4 * lg);
            f32x4 Y = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < 4; ++q) Y = mma_f32_k4(a[q], X[q], Y);
#pragma unroll
            for (int q = 0; q < 4; ++q) sT[(16 * i + 4 * lg + q) * L::LDA + 16 * j + li] = -Y[q];
        }
        lds_barrier();
    }
    // A is dead: V rows take its place (they waited in registers).
#pragma unroll
    for (int n = 0; n < NVV; ++n) {
        const int idx = tid + NT * n, r = idx / (DV / VE), cv = idx % (DV / VE);
        *(uint4 *)(sV + r * L::LDV + cv * VE) = vreg[n];
    }
    // Rows of T diag(c) (c = -beta e^g for -W, beta for U~) as 8-element
    // fragments, formed in registers from fp32 T: T[row][32 sk + 8 lg + e] c_s.
    // The blocks of T above its diagonal 16x16 blocks were never written and
    // are zero; with row = 32 m + p32_row(a, li) and sk = m they are the lanes
    // li < 8 with lg >= 2.
    f32x4 wsc[2][2], bsc[2][2];  // c_s for s = 32 sk + 8 lg + 4 h + q
#pragma unroll
    for (int sk = 0; sk < 2; ++sk)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            wsc[sk][hh] = *(const f32x4 *)(sw + 32 * sk + 8 * lg + 4 * hh);
            bsc[sk][hh] = *(const f32x4 *)(sb + 32 * sk + 8 * lg + 4 * hh);
        }
    lds_barrier();

    // -W fragments and Ut quads.  Wave w serves the two token tiles with
    // a_s = w & 1 (st = a_s, i.e. m = 0, and st = 2 + a_s, m = 1) and takes the
    // quarter q4 = w >> 1 of their outputs, so it forms the T diag(c) row
    // fragments of its tiles once -- three (m, s block) pairs, T being lower
    // triangular -- and shares the K^T and V fragments of s block 0 between
    // the two tiles.  Every wave issues the same number of MFMAs.
    static_assert(NWV == 8, "two token-tile parities x four quarters");
    const int as = w & 1, q4 = w >> 1;
    frag tw[3], tb[3];  // (m, sk) = (0, 0), (1, 0), (1, 1)
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        const int m = i > 0 ? 1 : 0, sk = i == 2 ? 1 : 0;
        const float *trow = sT + (32 * m + p32_row(as, li)) * L::LDA + 32 * sk + 8 * lg;
        f32x4 t0 = *(const f32x4 *)trow, t1 = *(const f32x4 *)(trow + 4);
        if (sk == m && lg >= 2 && li < 8) t0 = t1 = f32x4{0.f, 0.f, 0.f, 0.f};
        tw[i] = TR::cat(TR::from_f32(t0 * wsc[sk][0]), TR::from_f32(t1 * wsc[sk][1]));
        tb[i] = TR::cat(TR::from_f32(t0 * bsc[sk][0]), TR::from_f32(t1 * bsc[sk][1]));
    }
    // -W, computed transposed (W^T = K^T (T diag(beta e^g))^T) so that each lane
    // ends up holding the 8 consecutive Dk entries the scan consumes: fragment
    // f = (wave * 4 + st) * 2 + kb, lane (li, lg) =
    // -W[32 m + p32_row(a_s, li)][64 wave + 32 kb + 8 lg + e]  (st = 2 m + a_s).
    constexpr int NWC = NFR / 4;  // (wave, kb) combinations per token tile
    if (q4 < NWC) {
        const int wv = q4 >> 1, kb = q4 & 1, d0 = 64 * wv + 32 * kb;
        f32x4 w0[2], w1[2];  // tiles m = 0 and m = 1
#pragma unroll
        for (int a = 0; a < 2; ++a) {
            const frag k0 = tr_frag<E>(sK, L::LDK, 0, d0, true, a, li, lg);
            const frag k1 = tr_frag<E>(sK, L::LDK, 32, d0, true, a, li, lg);
            const f32x4 z = {0.f, 0.f, 0.f, 0.f};
            w0[a] = TR::mma(k0, tw[0], z);
            w1[a] = TR::mma(k1, tw[2], TR::mma(k0, tw[1], z));
        }
        E *Wf = p.W + cidx * (size_t)kChunk * DK + l * 8;
        TR::store8(Wf + ((wv * 4 + as) * 2 + kb) * 512, TR::cat(TR::from_f32(w0[0]), TR::from_f32(w0[1])));
        TR::store8(Wf + ((wv * 4 + 2 + as) * 2 + kb) * 512, TR::cat(TR::from_f32(w1[0]), TR::from_f32(w1[1])));
    }
    // Ut tiles (jt, st) in P32 row order, written as fragment-major quads
    // u = 4 jt + st: lane (li, lg) = Ut[32 m + 8 lg + 4 a_s + q][16 jt + li].
    constexpr int NJ = DV / 16;
    E *Uf = p.Ut + cidx * (size_t)DV * kChunk + l * 4;
#pragma unroll
    for (int j = 0; j < NJ / 4; ++j) {
        const int jt = q4 * (NJ / 4) + j;
        const frag v0 = tr_frag<E>(sV, L::LDV, 0, 16 * jt, false, 0, li, lg);
        const frag v1 = tr_frag<E>(sV, L::LDV, 32, 16 * jt, false, 0, li, lg);
        const f32x4 z = {0.f, 0.f, 0.f, 0.f};
        TR::store(Uf + (4 * jt + as) * 256, TR::from_f32(TR::mma(tb[0], v0, z)));
        TR::store(Uf + (4 * jt + 2 + as) * 256, TR::from_f32(TR::mma(tb[2], v1, TR::mma(tb[1], v0, z))));
    }
}

// --------------------------------------------------------------------------
// Stage 2: the state recurrence across chunks, H_c = gamma_c H_{c-1} + K_c^T D_c U_c
// with U_c = Ut_c - W_c H_{c-1} and D_c = diag(e^{g_C - g}), i.e.
// H_c = A_c H_{c-1} + B_c with the affine chunk transfer
// A_c = gamma_c I - K_c^T D_c W_c, B_c = K_c^T D_c Ut_c (the token-wise
// counterpart of the paper's S_f = alpha_f P_f S_{f-1} + A_f).  The chunks are
// cut into groups of G; the sequential dependency is reduced to one step per
// group:
//   (T) gdn_chunkscan_kernel<.., SCAN_TRANS>: for every group in parallel, run
//       the recurrence over its chunks from [Phi | Psi] = [I | 0], giving the
//       group transfer Phi_g = prod A_c and the zero-start state Psi_g;
//   (S) gdn_groupscan_kernel: H <- Phi_g H + Psi_g over the groups, recording
//       every group's entry state (and the final state);
//   (O) gdn_chunkscan_kernel<.., SCAN_STATES>: for every group in parallel, run
//       the recurrence from the group's true entry state and write the
//       per-chunk state H_{c-1} and pseudo-values U_c the output stage needs.
// With a single group only (O) runs, from state_in, and writes state_out.
//
// gdn_chunkscan_kernel: a workgroup owns NCW * 16 * CT state columns of one
// (b, h, group).  It has NCW compute waves, each carrying 16 * CT columns over
// all Dk rows through the group's chunks in fp32 accumulators (so U = Ut - W H
// needs no exchange between waves), and two loader waves that stream the chunk
// operands (-W, the chunk's key rows read from the input, the workgroup's Ut
// columns and the key scales e^{g_C - g}) into an LDS ring of DEPTH slots with
// asynchronous global->LDS copies (1 KB per instruction, lane i's 16 bytes
// landing at +16 i: the fragment-major workspace layout is kept, and each key
// row's 16-byte pieces land permuted, see kswz).  The update takes
// K^T (diag(e^{g_C - g}) U): the key scales are applied to U in registers.
// One workgroup barrier per chunk hands a slot over: before barrier c the
// loaders have waited (vmcnt) for chunk c's copies; after it they refill the
// slot of chunk c - 1, which every compute wave has finished reading.  The
// copies for chunk c are thus issued DEPTH - 1 chunks ahead, and neither the
// copy issue nor its latency sits on the compute waves' chain.
// --------------------------------------------------------------------------
enum { SCAN_TRANS = 0, SCAN_STATES = 1 };

// Column tiles per compute wave and compute waves per workgroup for the
// grouped passes; a single-group scan uses one column tile and one compute
// wave per workgroup (every workgroup loads all of W and K each chunk, so
// narrow workgroups spread that traffic over more CUs).
template <class E> struct ScanCT { static constexpr int value = sizeof(E) == 2 ? 2 : 1; };
constexpr int kScanNCW = 2;

template <class E, int DK, int CT, int NCW, bool FUSE = false> struct ScanLds {
    static constexpr int KB = DK / 32;                     // 32-row blocks of the state
    static constexpr int NT = DK / 16;                     // 16-row tiles of the state
    static constexpr int WK = kChunk * DK;                 // elements of -W (and of K) per chunk
    static constexpr int UT = NCW * CT * 1024;             // elements of the workgroup's Ut per chunk
    static constexpr int oD = 2 * WK + UT;                 // key scales, g_C: one gate record
    static constexpr int SLOT = oD + 4 * kGateRec / (int)sizeof(E);  // ring slot: -W, K rows, Ut, gates
    static constexpr int SLOT_BYTES = SLOT * (int)sizeof(E);
    static constexpr int NC_W = WK * (int)sizeof(E) / 1024;   // 1 KB copies of -W (and of K)
    static constexpr int NC_U = UT * (int)sizeof(E) / 1024;
    // loader 0 copies -W, the first half of Ut and the gate record (one
    // 17-lane copy), loader 1 the key rows and the rest of Ut
    static constexpr int NC_U0 = NC_U / 2, NC_U1 = NC_U - NC_U0;
    static constexpr int NCOPY0 = NC_W + NC_U0 + 1, NCOPY1 = NC_W + NC_U1;
    static constexpr int LDS_CAP = 152 * 1024;
    // fused output: H_{c-1} (KB fragments) and U (2) per column tile handed
    // from each compute wave to its output wave, double-buffered
    static constexpr int HOFF_FRAGS = CT * (KB + 2);
    static constexpr int HOFF_BYTES = FUSE ? 2 * NCW * HOFF_FRAGS * 64 * (int)sizeof(typename Tr<E>::frag) : 0;
    static constexpr int DL = (LDS_CAP - HOFF_BYTES) / SLOT_BYTES;
    // the loader waits with D - 2 younger chunks in flight: vmcnt <= 63
    static constexpr int DV_ = 2 + 63 / (NCOPY0 > NCOPY1 ? NCOPY0 : NCOPY1);
    static constexpr int DEPTH = (DL < 4 ? DL : 4) < DV_ ? (DL < 4 ? DL : 4) : DV_;
    static constexpr size_t oHOFF = (size_t)DEPTH * SLOT_BYTES;
    static constexpr size_t bytes = oHOFF + HOFF_BYTES;
    static_assert(DEPTH >= 2, "scan ring needs two slots");
    static_assert((WK * sizeof(E)) % 1024 == 0 && (UT * sizeof(E)) % 2048 == 0, "whole 1 KB copies");
};

// Copy N whole KB from global to LDS: instruction i moves bytes
// [1024 i, 1024 i + 1024), lane l its 16 bytes at 1024 i + 16 l.
template <int N> __device__ __forceinline__ void copy_kb(const void *src, void *dst, int l) {
#pragma unroll
    for (int i = 0; i < N; ++i)
        __builtin_amdgcn_global_load_lds((const void *)((const char *)src + 1024 * i + 16 * l),
                                         (__attribute__((address_space(3))) void *)((char *)dst + 1024 * i),
                                         16, 0, 0);
}

// Key rows in the scan's LDS ring: row r (a token of the chunk) holds its DK
// elements with the 16-byte granules permuted, granule g stored at g ^ kswz(r).
// The update's A operand is read with transposing reads, whose 16 lanes take
// 4 consecutive rows x 4 consecutive granules: the permutation sends them to
// 16 distinct bank groups.  kswz(r + 4) = kswz(r) for the rows r = 8 i + j,
// j < 4, those reads start from.  fp32 rows are gathered element by element
// and stay in order.
template <class E, int DK> __device__ __forceinline__ int kswz(int r) {
    constexpr int GPR = DK * (int)sizeof(E) / 16;  // granules per row
    if constexpr (sizeof(E) == 4)
        return 0;
    else if constexpr (GPR == 16)
        return 4 * (r & 3);         // 256-byte rows: the 4 rows take disjoint granule quads
    else
        return 4 * ((r >> 1) & 1);  // 128-byte rows: two per bank line, the pairs take disjoint quads
}

// Update A-operand fragment from the ring's key rows Kr (the tr_frag read in
// P32 order, through the permutation): lane (li, lg) receives
// K[row0 + 8 lg + q'][colbase + p32_row(a, li)], q' = 0..7.
template <class E, int DK>
__device__ __forceinline__ typename Tr<E>::frag kt_frag(const E *Kr, int row0, int colbase, int a, int li,
                                                        int lg) {
    if constexpr (sizeof(E) == 2) {
        typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
        const int row = row0 + 8 * lg + (li >> 2);
        const int off = 8 * ((colbase / 8 + (li & 3)) ^ kswz<E, DK>(row)) + 4 * a;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(Kr + row * DK + off));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(Kr + (row + 4) * DK + off));
        return Tr<E>::cat(__builtin_bit_cast(u32x2, lo), __builtin_bit_cast(u32x2, hi));
    } else {
        return tr_frag<E>(Kr, DK, row0, colbase, true, a, li, lg);
    }
}

template <class E, int DK, int DV, int PHASE, int CT, int NCW, bool FUSE = false>
__global__ __launch_bounds__((NCW * (FUSE ? 2 : 1) + 2) * 64) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gdn_chunkscan_kernel(Params<E> p) {
    using TR = Tr<E>;
    using frag = typename TR::frag;
    using L = ScanLds<E, DK, CT, NCW, FUSE>;
    static_assert(!FUSE || PHASE == SCAN_STATES, "the output is fused into the state pass only");
    constexpr int NOW = FUSE ? NCW : 0;                  // output waves
    constexpr int D = L::DEPTH;
    // compute waves read the next chunk's operands ahead when the ring has
    // room for it (four slots: the loaders then still issue two chunks ahead)
    constexpr int AHEAD = D >= 4 ? 1 : 0;
    constexpr int KB = L::KB, NT = L::NT;
    constexpr int WGC = NCW * 16 * CT;                   // columns per workgroup
    constexpr int WCOLS = PHASE == SCAN_TRANS ? DK + DV : DV;
    constexpr int NJB = WCOLS / WGC;                     // column blocks per (b, h, group)
    static_assert(WCOLS % WGC == 0 && DK % WGC == 0, "column blocks do not straddle Phi and Psi");
    extern __shared__ __align__(16) unsigned char scan_lds[];
    E *ring = (E *)scan_lds;

    // XCD-aware placement: workgroups are dealt round-robin to the 8 XCDs, so
    // id = 8 slot + x runs on XCD x.  The NJB column blocks of one (b, h, group)
    // get consecutive slots of the same XCD and share its L2 for the chunk
    // operands W, K that all of them read.
    const int id = blockIdx.x, x = id & 7, slot = id >> 3;
    const int unit = (slot / NJB) * 8 + x, jb = slot % NJB;
    if (unit >= p.B * p.H * p.NG) return;
    const int bh = unit / p.NG, grp = unit - bh * p.NG;
    const int b = bh / p.H, h = bh - b * p.H;
    const int c_begin = grp * p.G, c_end = min(p.NC, c_begin + p.G);
    // w is wave-uniform: scalar branches and addresses
    const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), l = tid & 63, li = l & 15,
              lg = l >> 4;
    const int col0 = WGC * jb;
    const bool is_phi = PHASE == SCAN_TRANS && col0 < DK;
    // first column of this workgroup within the state (Phi columns or Psi / H columns)
    const int wbase = (PHASE == SCAN_TRANS && !is_phi) ? col0 - DK : col0;
    const bool has_ut = PHASE == SCAN_STATES || !is_phi;
    auto slot_of = [&](int c) { return ring + (size_t)((c - c_begin) % D) * L::SLOT; };

    // fused output hand-off: buffer i, compute wave wc, fragment f of column tile ct
    frag *hoff = (frag *)(scan_lds + L::oHOFF);
    auto hoff_at = [&](int i, int wc, int ct, int f) {
        return hoff + ((size_t)((i * NCW + wc) * CT + ct) * (KB + 2) + f) * 64 + l;
    };

    if (w >= NCW + NOW) {
        // ---------------- loader waves ----------------
        const int ld = w - NCW - NOW;
        // Key rows of chunk `src` from the input (B, T, H, DK): instruction n,
        // lane l fills LDS granule 64 n + l, i.e. granule (64 n + l) % GPR of
        // row (64 n + l) / GPR, from the row's granule permuted back by kswz.
        // Rows past the sequence's end are read from its last token; their
        // pseudo-values are exactly zero (beta = 0 and zero V and K rows in the
        // WY factors), so they add nothing to the update.
        auto copy_krows = [&](int src, E *dst) {
            constexpr int GPR = DK * (int)sizeof(E) / 16, VE = 16 / (int)sizeof(E);
            const int t0 = src * kChunk, tl = p.T - 1;
            const E *kbase = p.k + (size_t)b * p.T * p.H * DK + (size_t)h * DK;
#pragma unroll
            for (int n = 0; n < L::NC_W; ++n) {
                const int idx = 64 * n + l, r = idx / GPR, g = (idx % GPR) ^ kswz<E, DK>(r);
                const int t = min(t0 + r, tl);
                __builtin_amdgcn_global_load_lds((const void *)(kbase + (size_t)t * p.H * DK + g * VE),
                                                 (__attribute__((address_space(3))) void *)((char *)dst + 1024 * n),
                                                 16, 0, 0);
            }
        };
        // copies of chunk `src` into the slot of chunk `dst` (dst = src except
        // past the end, see below)
        auto issue = [&](int dst, int src) {
            const size_t cidx = (size_t)bh * p.NC + src;
            E *sl = slot_of(dst);
            const E *ut = p.Ut + cidx * (size_t)DV * kChunk + (size_t)(wbase / 16) * 1024;
            if (ld == 0) {
                copy_kb<L::NC_W>(p.W + cidx * (size_t)L::WK, sl, l);
                if (has_ut) copy_kb<L::NC_U0>(ut, sl + 2 * L::WK, l);
                if (l < kGateRec / 4)  // the gate record: 272 bytes
                    __builtin_amdgcn_global_load_lds((const void *)(p.gf + cidx * kGateRec + 4 * l),
                                                     (__attribute__((address_space(3))) void *)(sl + L::oD), 16, 0,
                                                     0);
            } else {
                copy_krows(src, sl + L::WK);
                if (has_ut)
                    copy_kb<L::NC_U1>((const char *)ut + 1024 * L::NC_U0,
                                      (char *)(sl + 2 * L::WK) + 1024 * L::NC_U0, l);
            }
        };
        // Chunk c (with AHEAD chunk c + 1) has landed once at most D - 2
        // (D - 3) younger chunks' copies are in flight (every chunk issues the
        // same number of copies).
        constexpr int NF = D - 2 - AHEAD;
        auto wait_oldest = [&]() {
            if (ld == 0) {
                if (has_ut) wait_vmcnt<NF * L::NCOPY0>();
                else wait_vmcnt<NF * (L::NC_W + 1)>();
            } else {
                if (has_ut) wait_vmcnt<NF * L::NCOPY1>();
                else wait_vmcnt<NF * L::NC_W>();
            }
        };
        // Prologue: chunks c_begin .. c_begin + D - 2.  Past the end the loaders
        // still issue the same number of copies (so that the per-chunk count the
        // waits rely on is constant), reading the last chunk, into the slot of
        // the missing chunk: a slot no compute wave reads again.
#pragma unroll
        for (int i = 0; i < D - 1; ++i) issue(c_begin + i, min(c_begin + i, c_end - 1));
        for (int c = c_begin; c < c_end; ++c) {
            wait_oldest();
            lds_only_barrier();  // chunk c handed to the compute waves
            // refills the slot of chunk c - 1
            issue(c + D - 1, min(c + D - 1, c_end - 1));
        }
        wait_vmcnt<0>();
        lds_only_barrier();                     // ring quiet: the compute waves may reuse it
        if (PHASE == SCAN_TRANS && is_phi) lds_only_barrier();  // matches the N staging barrier
        return;
    }

    if constexpr (FUSE) {
        if (w >= NCW) {
            // ---------------- output waves ----------------
            // Output wave wo finishes chunk c - 1 after barrier c (and the
            // last chunk after the final barrier) for the columns of compute
            // wave wo:  O^T = H_{c-1}^T Qf^T + U^T Pf^T, per token tile rt
            //   A operands: the handed-off H_{c-1} and U fragments (B-operand
            //   layout over d, resp. s, which is also the A layout),
            //   B operands: the Qf / Pf row fragments of the chunk.
            // Lane (li, lg) gets O[16 rt + li][jw + 16 ct + 4 lg + q].
            const int wo = w - NCW;
            const int jw = wbase + 16 * CT * wo;
            // Operands of chunk c live in register set (c - c_begin) & 1: at
            // barrier c the wave requests chunk c's and finishes chunk c - 1
            // from the other set, so a load is consumed one chunk later.
            frag q0[4][KB], p0[4][2], q1[4][KB], p1[4][2];
            auto load_ops = [&](int c, frag (&q)[4][KB], frag (&pf)[4][2]) {
                const size_t cidx = (size_t)bh * p.NC + c;
                const E *Qf = p.Qf + cidx * (size_t)kChunk * DK + l * 8;
                const E *Pf = p.Pf + cidx * (size_t)kChunk * kChunk + l * 8;
#pragma unroll
                for (int rt = 0; rt < 4; ++rt) {
#pragma unroll
                    for (int kb = 0; kb < KB; ++kb) q[rt][kb] = TR::load8(Qf + (size_t)(rt * KB + kb) * 512);
#pragma unroll
                    for (int m = 0; m < 2; ++m)
                        if (m == 0 || rt >= 2) pf[rt][m] = TR::load8(Pf + (size_t)(rt * 2 + m) * 512);
                }
            };
            auto finish = [&](int c, const frag (&cq)[4][KB], const frag (&cp)[4][2]) {
                const int i = (c - c_begin) & 1;
                const int nvalid = min(kChunk, p.T - c * kChunk);
                const size_t row0 = ((size_t)b * p.T + (size_t)c * kChunk) * p.H + h;
#pragma unroll
                for (int ct = 0; ct < CT; ++ct) {
                    frag hbf[KB], ubf[2];
#pragma unroll
                    for (int f = 0; f < KB; ++f) hbf[f] = *hoff_at(i, wo, ct, f);
#pragma unroll
                    for (int m = 0; m < 2; ++m) ubf[m] = *hoff_at(i, wo, ct, KB + m);
#pragma unroll
                    for (int rt = 0; rt < 4; ++rt) {
                        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                        for (int kb = 0; kb < KB; ++kb) acc = TR::mma(hbf[kb], cq[rt][kb], acc);
#pragma unroll
                        for (int m = 0; m < 2; ++m)
                            if (m == 0 || rt >= 2) acc = TR::mma(ubf[m], cp[rt][m], acc);
                        const int r = 16 * rt + li;
                        if (r < nvalid)
                            TR::store(p.out + (row0 + (size_t)r * p.H) * DV + jw + 16 * ct + 4 * lg, TR::from_f32(acc));
                    }
                }
            };
            for (int c = c_begin; c < c_end; c += 2) {
                lds_only_barrier();  // barrier c
                load_ops(c, q0, p0);
                if (c > c_begin) finish(c - 1, q1, p1);
                if (c + 1 < c_end) {
                    lds_only_barrier();  // barrier c + 1
                    load_ops(c + 1, q1, p1);
                    finish(c, q0, p0);
                }
            }
            lds_only_barrier();  // the compute waves have handed off the last chunk
            if ((c_end - 1 - c_begin) & 1)
                finish(c_end - 1, q1, p1);
            else
                finish(c_end - 1, q0, p0);
            return;
        }
    }

    // ---------------- compute waves ----------------
    const int jw = wbase + 16 * CT * w;          // this wave's first column
    // State H[:, jw + 16 ct + li] as NT accumulator tiles in P32 order:
    // Hacc[t][ct][q] = H[32 (t / 2) + 8 lg + 4 (t % 2) + q][jw + 16 ct + li].
    f32x4 Hacc[NT][CT];
    auto row0 = [&](int t) { return 32 * (t >> 1) + 8 * lg + 4 * (t & 1); };
    if constexpr (PHASE == SCAN_TRANS) {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    Hacc[t][ct][q] = (is_phi && row0(t) + q == jw + 16 * ct + li) ? 1.f : 0.f;
    } else if (p.NG > 1) {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int t = 0; t < NT; ++t)
                Hacc[t][ct] = *(const f32x4 *)(p.HgT + ((size_t)unit * DV + jw + 16 * ct + li) * DK + row0(t));
    } else if (p.state_in) {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    Hacc[t][ct][q] = p.state_in[((size_t)bh * DK + row0(t) + q) * DV + jw + 16 * ct + li];
    } else {
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int t = 0; t < NT; ++t) Hacc[t][ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    double lgam = 0.0;  // sum of gC over the group

    // Operands of one chunk, read from its ring slot (fragment layouts below).
    // With AHEAD the wave reads chunk c + 1's slot while it computes chunk c,
    // so the LDS latency stays off the chain.
    struct Ops {
        frag wf[KB][4], kf[NT][2];
        typename TR::quad us[4][CT];
        f32x4 dsc[4];
        double gC;
        float gam;
    };
    //   -W fragment (wave kb / 2, token tile st, k block kb % 2),
    //   K^T fragment (row tile t, token block m): rows d in P32 order
    //     32 (t / 2) + p32_row(t % 2, li), tokens 32 m + 8 lg + e,
    //   U~t quad of token tile st = 2 m + a: tokens 32 m + 8 lg + 4 a + q
    //     (zero for Phi columns), and the key scales of the same tokens,
    //   g_C and gamma = e^{g_C} (broadcast reads).
    auto read_ops = [&](int c, Ops &o) {
        const E *sl = slot_of(c);
        const float *Dl = (const float *)(sl + L::oD);
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int st = 0; st < 4; ++st)
                o.us[st][ct] = has_ut ? TR::load(sl + 2 * L::WK + (size_t)w * CT * 1024 + l * 4 + ct * 1024 + st * 256)
                                      : TR::zero();
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int a = 0; a < 2; ++a) {
                    const int st = 2 * m + a;
                    o.wf[kb][st] = TR::load8(sl + l * 8 + (((kb >> 1) * 4 + st) * 2 + (kb & 1)) * 512);
                }
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int t = 0; t < NT; ++t)
                o.kf[t][m] = kt_frag<E, DK>(sl + L::WK, 32 * m, 32 * (t >> 1), t & 1, li, lg);
#pragma unroll
        for (int st = 0; st < 4; ++st) o.dsc[st] = *(const f32x4 *)(Dl + 32 * (st >> 1) + 8 * lg + 4 * (st & 1));
        o.gC = *(const double *)(Dl + kChunk);
        o.gam = Dl[kChunk + 2];
    };

    // bf16: the U~t seeds enter the accumulators through an MFMA with a 0/1
    // selection operand (exact: one product 1 x u per entry), so no VALU
    // unpacking sits before the first W H MFMA.  sel[a] places the 32-token
    // B fragment cat(us[2 m], us[2 m + 1]) (lane (li, lg): tokens 32 m + 8 lg
    // + e') in the rows of tile 2 m + a, i.e. tile row i takes token
    // 32 m + p32_row(a, i): lane (li, lg) of sel[a] holds 1 at e' = 4 a +
    // li % 4 when lg = li / 4, else 0.
    frag sel[2];
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        f32x4 lo = {0.f, 0.f, 0.f, 0.f}, hi = {0.f, 0.f, 0.f, 0.f};
        if (lg == (li >> 2)) {
            if (a == 0) lo[li & 3] = 1.f;
            else hi[li & 3] = 1.f;
        }
        sel[a] = TR::cat(TR::from_f32(lo), TR::from_f32(hi));
    }

    // One chunk: U = U~t - W H_{c-1} (the workspace holds -W), then
    // H_c = gamma H_{c-1} + K^T (diag(e^{g_C - g}) U).  The chain per token
    // half m: its W H MFMAs, the conversion of its U half (as is, for the
    // output, and scaled by e^{g_C - g}, for the update), then that half's
    // update.  Half 0 is finished first, so its conversion overlaps the MFMAs
    // of half 1, and half 1's conversion those of the first update.  The
    // output wave's operands (H_{c-1}, then each U half) are handed off as
    // soon as they exist, so the stores have drained by the next barrier.
    auto step = [&](int c, const Ops &o) {
        const size_t cidx = (size_t)bh * p.NC + c;
        const int i = (c - c_begin) & 1;
        // H_{c-1} rounded to E: B operands over the KB 32-row blocks.
        frag hb[KB][CT];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) {
                hb[kb][ct] = TR::cat(TR::from_f32(Hacc[2 * kb][ct]), TR::from_f32(Hacc[2 * kb + 1][ct]));
                if constexpr (FUSE) *hoff_at(i, w, ct, kb) = hb[kb][ct];
            }
        lgam += o.gC;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) Hacc[t][ct] *= o.gam;
        f32x4 part[4][CT];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int st = 0; st < 4; ++st) {
                if constexpr (sizeof(E) == 2)
                    part[st][ct] = TR::mma(sel[st & 1], TR::cat(o.us[st & 2][ct], o.us[(st & 2) + 1][ct]),
                                           f32x4{0.f, 0.f, 0.f, 0.f});
                else
                    part[st][ct] = TR::to_f32(o.us[st][ct]);
            }
        frag ub[2][CT], uk[2][CT];
        auto wh_half = [&](int m) {
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int a = 0; a < 2; ++a)
#pragma unroll
                    for (int ct = 0; ct < CT; ++ct)
                        part[2 * m + a][ct] = TR::mma(o.wf[kb][2 * m + a], hb[kb][ct], part[2 * m + a][ct]);
        };
        auto cvt_half = [&](int m) {
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                ub[m][ct] = TR::cat(TR::from_f32(part[2 * m][ct]), TR::from_f32(part[2 * m + 1][ct]));
                uk[m][ct] = TR::cat(TR::from_f32(part[2 * m][ct] * o.dsc[2 * m]),
                                    TR::from_f32(part[2 * m + 1][ct] * o.dsc[2 * m + 1]));
                if constexpr (FUSE) *hoff_at(i, w, ct, KB + m) = ub[m][ct];
            }
        };
        auto kt_half = [&](int m) {
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int ct = 0; ct < CT; ++ct) Hacc[t][ct] = TR::mma(o.kf[t][m], uk[m][ct], Hacc[t][ct]);
        };
        wh_half(0);
        wh_half(1);
        cvt_half(0);
        kt_half(0);
        cvt_half(1);
        kt_half(1);
        if constexpr (PHASE == SCAN_STATES && !FUSE) {
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
#pragma unroll
                for (int kb = 0; kb < KB; ++kb)
                    TR::store8(p.Hs + cidx * (size_t)DV * DK + (size_t)(jw + 16 * ct + li) * DK + 32 * kb + 8 * lg,
                               hb[kb][ct]);
                E *Us = p.Us + cidx * (size_t)DV * kChunk + (size_t)(jw + 16 * ct + li) * kChunk + 8 * lg;
                TR::store8(Us, ub[0][ct]);
                TR::store8(Us + 32, ub[1][ct]);
            }
        }
    };

    // Barrier c hands over chunk c (and, with AHEAD, chunk c + 1: the loaders
    // wait one chunk further).  Operand sets alternate between chunks.
    Ops opA, opB;
    for (int c = c_begin; c < c_end; c += 2) {
        lds_only_barrier();  // barrier c
        if constexpr (AHEAD) {
            if (c == c_begin) read_ops(c, opA);
            read_ops(c + 1, opB);  // past the end: a padding slot, not used
        } else {
            read_ops(c, opA);
        }
        step(c, opA);
        if (c + 1 >= c_end) break;
        lds_only_barrier();  // barrier c + 1
        if constexpr (AHEAD)
            read_ops(c + 2, opA);
        else
            read_ops(c + 1, opB);
        step(c + 1, opB);
    }
    lds_only_barrier();  // the loaders have drained: the ring is free

    const size_t gidx = (size_t)bh * p.NG + grp;
    if constexpr (PHASE == SCAN_STATES) {
        if (p.NG == 1 && p.state_out) {
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                for (int t = 0; t < NT; ++t)
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        p.state_out[((size_t)bh * DK + row0(t) + q) * DV + jw + 16 * ct + li] = Hacc[t][ct][q];
        }
    } else if (!is_phi) {  // SCAN_TRANS from here on
        // Psi_g^T [Dv][Dk], fp32
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
#pragma unroll
            for (int t = 0; t < NT; ++t)
                *(f32x4 *)(p.PsiT + (gidx * DV + jw + 16 * ct + li) * DK + row0(t)) = Hacc[t][ct];
    } else {
        if (jb == 0 && w == 0 && l == 0) p.lgam[gidx] = lgam;
        // N_g = Phi_g - Gamma_g I, rounded to E, staged in LDS (in the ring
        // memory) as N^T (row e = state column - col0, rows d contiguous) and
        // re-read with the transposing LDS read into the group scan's A-operand
        // fragments: fragment (wave v, row tile t, k block kb), lane (li, lg) =
        //   N[64 v + 32 (t / 2) + p32_row(t % 2, li)][32 kb + 8 lg + e].
        static_assert(WGC % 32 == 0, "the transfer pass writes whole 32-column k blocks");
        constexpr int LDN = DK + 16 / (int)sizeof(E);
        static_assert(sizeof(E) * WGC * LDN <= L::bytes, "N^T staging");
        const float Gam = expf((float)lgam);
        E *sN = ring;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
            const int e = 16 * CT * w + 16 * ct + li;  // staging row
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) {
                f32x4 lo = Hacc[2 * kb][ct], hi = Hacc[2 * kb + 1][ct];
                const int r0 = 32 * kb + 8 * lg;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (r0 + q == col0 + e) lo[q] -= Gam;
                    if (r0 + 4 + q == col0 + e) hi[q] -= Gam;
                }
                TR::store8(sN + e * LDN + r0, TR::cat(TR::from_f32(lo), TR::from_f32(hi)));
            }
        }
        lds_only_barrier();  // staging written (the loaders take this barrier too)
        const int kb0 = col0 / 32;
        constexpr int NKB = WGC / 32;                       // k blocks in this workgroup
        constexpr int NFRAG = (DK / 64) * 4 * NKB;
        E *Nf = p.Nf + gidx * (size_t)DK * DK + l * 8;
        for (int f = w; f < NFRAG; f += NCW) {
            const int v = f / (4 * NKB), t = (f / NKB) % 4, kk = f % NKB;
            const frag nf = tr_frag<E>(sN, LDN, 32 * kk, 64 * v + 32 * (t >> 1), true, t & 1, li, lg);
            TR::store8(Nf + (size_t)((v * 4 + t) * (DK / 32) + kb0 + kk) * 512, nf);
        }
    }
}

// --------------------------------------------------------------------------
// Group scan: H <- Gamma_g H + N_g H + Psi_g over the groups of one (b, h), in
// 16-column blocks (one workgroup each, Dk/64 waves splitting the rows, which
// exchange their halves of H each step through LDS).  Records every group's
// entry state H^T for the state stage and writes the final state.
// --------------------------------------------------------------------------
template <class E, int DK, int DV>
__global__ __launch_bounds__(DK) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gdn_groupscan_kernel(Params<E> p) {
    using TR = Tr<E>;
    using frag = typename TR::frag;
    constexpr int NW = DK / 64;
    constexpr int NJ = DV / 16;
    constexpr int KB = DK / 32;
    __shared__ frag sH[2][NW][2][64];  // bf16 halves of H, double-buffered

    const int id = blockIdx.x, x = id & 7, slot = id >> 3;
    const int bh = (slot / NJ) * 8 + x, jt = slot % NJ;
    if (bh >= p.B * p.H) return;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lg = l >> 4;
    const int d0 = 64 * w;
    const int j = 16 * jt + li;

    f32x4 Hacc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            Hacc[t][q] = p.state_in ? p.state_in[((size_t)bh * DK + d0 + 32 * (t >> 1) + 8 * lg +
                                                  4 * (t & 1) + q) * DV + j]
                                    : 0.f;
    frag nf[4][KB];
    f32x4 ps[4];
    double lg_g;
    auto fetch = [&](int g) {
        const size_t gidx = (size_t)bh * p.NG + g;
        const E *Nc = p.Nf + gidx * (size_t)DK * DK + (size_t)w * 4 * KB * 512 + l * 8;
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) nf[t][kb] = TR::load8(Nc + (t * KB + kb) * 512);
#pragma unroll
        for (int t = 0; t < 4; ++t)
            ps[t] = *(const f32x4 *)(p.PsiT + (gidx * DV + j) * DK + d0 + 32 * (t >> 1) + 8 * lg + 4 * (t & 1));
        lg_g = p.lgam[gidx];
    };
    fetch(0);
    for (int g = 0; g < p.NG; ++g) {
        const size_t gidx = (size_t)bh * p.NG + g;
        // entry state of group g
#pragma unroll
        for (int t = 0; t < 4; ++t)
            *(f32x4 *)(p.HgT + (gidx * DV + j) * DK + d0 + 32 * (t >> 1) + 8 * lg + 4 * (t & 1)) = Hacc[t];
        frag hb[KB];
        const frag own0 = TR::cat(TR::from_f32(Hacc[0]), TR::from_f32(Hacc[1]));
        const frag own1 = TR::cat(TR::from_f32(Hacc[2]), TR::from_f32(Hacc[3]));
        if constexpr (NW > 1) {
            const int buf = g & 1;
            sH[buf][w][0][l] = own0;
            sH[buf][w][1][l] = own1;
            lds_barrier();
            hb[2 * w] = own0;
            hb[2 * w + 1] = own1;
            hb[2 * (1 - w)] = sH[buf][1 - w][0][l];
            hb[2 * (1 - w) + 1] = sH[buf][1 - w][1][l];
        } else {
            hb[0] = own0;
            hb[1] = own1;
        }
        const float Gam = expf((float)lg_g);
#pragma unroll
        for (int t = 0; t < 4; ++t) Hacc[t] = Hacc[t] * Gam + ps[t];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int t = 0; t < 4; ++t) Hacc[t] = TR::mma(nf[t][kb], hb[kb], Hacc[t]);
        fetch(min(g + 1, p.NG - 1));
    }
    if (p.state_out) {
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                p.state_out[((size_t)bh * DK + d0 + 32 * (t >> 1) + 8 * lg + 4 * (t & 1) + q) * DV + j] =
                    Hacc[t][q];
    }
}

// --------------------------------------------------------------------------
// Stage 3: per-chunk output.  Grid (NC, B*H), 256 threads; wave w produces
// tokens 16w..16w+15 of the chunk for all Dv columns, as O^T tiles:
//   O^T = H_{c-1}^T Q^T diag(e^g) + U^T P^T,   P^T[s][r] = e^{g_r-g_s} k_s.q_r (s <= r)
// --------------------------------------------------------------------------
template <class E, int DK, int DV> struct OutLds {
    static constexpr int PAD = 16 / (int)sizeof(E);
    static constexpr int LDH = DK + PAD;
    static constexpr int LDU = kChunk + PAD;
    static constexpr int LDK = DK + PAD;
    static constexpr size_t oH = 0;
    static constexpr size_t oU = oH + sizeof(E) * DV * LDH;
    static constexpr size_t oK = oU + sizeof(E) * DV * LDU;
    static constexpr size_t oG = oK + sizeof(E) * kChunk * LDK;
    static constexpr size_t bytes = oG + 8 * kChunk;
};

template <class E, int DK, int DV>
__global__ __launch_bounds__(256) void gdn_output_kernel(Params<E> p) {
    using L = OutLds<E, DK, DV>;
    using TR = Tr<E>;
    using frag = typename TR::frag;
    using quad = typename TR::quad;
    constexpr int VE = 16 / (int)sizeof(E);            // elements per 16-byte vector
    constexpr int NH = DV * DK / VE / 256;             // H^T vectors per thread
    constexpr int NU = DV * kChunk / VE / 256;         // U^T vectors per thread
    constexpr int NK = kChunk * DK / VE / 256;         // K vectors per thread
    extern __shared__ __align__(16) unsigned char smem[];
    E *sH = (E *)(smem + L::oH);
    E *sU = (E *)(smem + L::oU);
    E *sK = (E *)(smem + L::oK);
    double *sg = (double *)(smem + L::oG);

    const int c = blockIdx.x, bh = blockIdx.y;
    const int b = bh / p.H, h = bh - b * p.H;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lg = l >> 4;
    const int t0 = c * kChunk;
    const int nvalid = min(kChunk, p.T - t0);
    const size_t cidx = (size_t)bh * p.NC + c;
    const size_t row0 = ((size_t)b * p.T + t0) * p.H + h;
    const size_t rstride = (size_t)p.H;

    // Every global load is issued before the first LDS store, so their
    // latencies overlap: Q rows of this wave's tokens as B operands
    // (B[k=d][n=r] = Q[r][d]; padded tokens are 0), then H^T, U^T and K
    // rows with 16-byte coalesced loads.
    const int r = 16 * w + li;  // token within the chunk
    const bool rvalid = r < nvalid;
    frag qf[DK / 32];
#pragma unroll
    for (int kb = 0; kb < DK / 32; ++kb)
        qf[kb] = rvalid ? load_frag<E>(p.q + (row0 + r * rstride) * DK + 32 * kb, lg) : TR::cat(TR::zero(), TR::zero());
    uint4 hreg[NH], ureg[NU], kreg[NK];
    const E *Hs = p.Hs + cidx * (size_t)DV * DK;
    const E *Us = p.Us + cidx * (size_t)DV * kChunk;
#pragma unroll
    for (int n = 0; n < NH; ++n) hreg[n] = *(const uint4 *)(Hs + (size_t)(tid + 256 * n) * VE);
#pragma unroll
    for (int n = 0; n < NU; ++n) ureg[n] = *(const uint4 *)(Us + (size_t)(tid + 256 * n) * VE);
#pragma unroll
    for (int n = 0; n < NK; ++n) {
        const int idx = tid + 256 * n, kr = idx / (DK / VE), kc = idx % (DK / VE);
        kreg[n] = kr < nvalid ? *(const uint4 *)(p.k + (row0 + kr * rstride) * DK + kc * VE) : make_uint4(0u, 0u, 0u, 0u);
    }
    if (tid < kChunk) sg[tid] = p.g[cidx * kChunk + tid];
#pragma unroll
    for (int n = 0; n < NH; ++n) {
        const int idx = tid + 256 * n;
        *(uint4 *)(sH + (idx / (DK / VE)) * L::LDH + (idx % (DK / VE)) * VE) = hreg[n];
    }
#pragma unroll
    for (int n = 0; n < NU; ++n) {
        const int idx = tid + 256 * n;
        *(uint4 *)(sU + (idx / (kChunk / VE)) * L::LDU + (idx % (kChunk / VE)) * VE) = ureg[n];
    }
#pragma unroll
    for (int n = 0; n < NK; ++n) {
        const int idx = tid + 256 * n;
        *(uint4 *)(sK + (idx / (DK / VE)) * L::LDK + (idx % (DK / VE)) * VE) = kreg[n];
    }
    lds_barrier();

    // P^T tiles in P32 order (tile st = 2 m + a holds tokens 32 m + p32_row(a, i)),
    // masked (s <= r) and decayed, rounded to E.  Block m = 1 only matters for r >= 32.
    const double gr = sg[r];
    quad pq[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
        const int m = st >> 1, a = st & 1;
        pq[st] = TR::zero();
        if (m == 0 || w >= 2) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < DK / 32; ++kb)
                acc = TR::mma(load_frag<E>(sK + (32 * m + p32_row(a, li)) * L::LDK + 32 * kb, lg),
                              qf[kb], acc);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int s2 = 32 * m + 8 * lg + 4 * a + q;
                acc[q] = (s2 <= r) ? expf((float)(gr - sg[s2])) * acc[q] : 0.f;
            }
            pq[st] = TR::from_f32(acc);
        }
    }
    const frag pf0 = TR::cat(pq[0], pq[1]);
    const frag pf1 = TR::cat(pq[2], pq[3]);
    const float er = expf((float)gr);

    // O^T = H^T Q^T e^{g_r} + U^T P^T in 32-column blocks J; the two tiles a of
    // a block take A rows (output columns) 32 J + p32_row(a, i), so lane
    // (li, lg) ends up with the 8 consecutive columns 32 J + 8 lg + [0, 8) of
    // token r and writes them with one 16-byte store.
    E *orow = p.out + (row0 + r * rstride) * DV;
#pragma unroll 2
    for (int J = 0; J < DV / 32; ++J) {
        f32x4 acc[2];
#pragma unroll
        for (int a = 0; a < 2; ++a) {
            const int col = 32 * J + p32_row(a, li);
            f32x4 x = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < DK / 32; ++kb)
                x = TR::mma(load_frag<E>(sH + col * L::LDH + 32 * kb, lg), qf[kb], x);
            x *= er;
            x = TR::mma(load_frag<E>(sU + col * L::LDU, lg), pf0, x);
            if (w >= 2) x = TR::mma(load_frag<E>(sU + col * L::LDU + 32, lg), pf1, x);
            acc[a] = x;
        }
        if (rvalid) TR::store8(orow + 32 * J + 8 * lg, TR::cat(TR::from_f32(acc[0]), TR::from_f32(acc[1])));
    }
}

}  // namespace gdn
