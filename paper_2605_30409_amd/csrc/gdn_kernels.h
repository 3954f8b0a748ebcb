// The three gfx950 kernels of the GDN chunk forward.
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
//   W  [64][Dk]   E      WY factor, token-major
//   Kt [Dk][64]   E      (diag(e^{g_C - g}) K)^T
//   Ut [Dv][64]   E      Ut^T
//   Hs [Dv][Dk]   E      H_{c-1}^T, the state entering the chunk
//   Us [Dv][64]   E      U^T
#pragma once

#include "gdn_device.h"

namespace gdn {

template <class E> struct Params {
    const E *q, *k, *v;
    const float *alpha, *beta, *state_in;
    E *out;
    float *state_out;
    int B, H, T, NC;
    double *g;
    E *W, *Kt, *Ut, *Hs, *Us;
};

constexpr float kLogAlphaMin = -87.3f;  // ~ log(FLT_MIN): alpha below this acts as 1.2e-38

// --------------------------------------------------------------------------
// Stage 1: per-chunk WY / UT transform.  Grid (NC, B*H), 256 threads.
// --------------------------------------------------------------------------
template <class E, int DK, int DV> struct WyLds {
    static constexpr int PAD = 16 / (int)sizeof(E);
    static constexpr int LDK = DK + PAD;      // K (row-major), later the W staging tile
    static constexpr int LDT = kChunk + PAD;  // K^T and V^T (token-contiguous rows)
    static constexpr int LDA = kChunk + 4;    // A and T (fp32)
    static constexpr size_t szA = 4 * kChunk * LDA;
    static constexpr size_t szVt = sizeof(E) * DV * LDT;
    static constexpr size_t oK = 0;
    static constexpr size_t oKt = oK + sizeof(E) * kChunk * LDK;
    static constexpr size_t oA = oKt + sizeof(E) * DK * LDT;     // A, then V^T once A is dead
    static constexpr size_t oT = oA + (szA > szVt ? szA : szVt);
    static constexpr size_t oG = oT + szA;
    static constexpr size_t bytes = oG + 8 * kChunk + 4 * 3 * kChunk;
};

template <class E, int DK, int DV>
__global__ __launch_bounds__(256) void gdn_wy_kernel(Params<E> p) {
    using L = WyLds<E, DK, DV>;
    using TR = Tr<E>;
    constexpr int VE = 16 / (int)sizeof(E);   // elements per 16-byte vector
    constexpr int NVV = kChunk * (DV / VE) / 256;
    extern __shared__ __align__(16) unsigned char smem[];
    E *sK = (E *)(smem + L::oK);
    E *sKt = (E *)(smem + L::oKt);
    float *sA = (float *)(smem + L::oA);
    E *sVt = (E *)(smem + L::oA);
    float *sT = (float *)(smem + L::oT);
    double *sg = (double *)(smem + L::oG);     // g_r
    float *sb = (float *)(sg + kChunk);        // beta_r
    float *sw = sb + kChunk;                   // beta_r e^{g_r}
    float *sd = sw + kChunk;                   // e^{g_C - g_r}

    const int c = blockIdx.x, bh = blockIdx.y;
    const int b = bh / p.H, h = bh - b * p.H;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lg = l >> 4;
    const int t0 = c * kChunk;
    const int nvalid = min(kChunk, p.T - t0);
    const size_t cidx = (size_t)bh * p.NC + c;
    const size_t row0 = ((size_t)b * p.T + t0) * p.H + h;  // token-row index of token t0
    const size_t rstride = (size_t)p.H;                    // token-row stride

    // V is only needed after the solve; its loads are issued now (lane = token row).
    uint4 vreg[NVV];
#pragma unroll
    for (int n = 0; n < NVV; ++n) {
        const int cv = w + 4 * n;
        vreg[n] = make_uint4(0u, 0u, 0u, 0u);
        if (l < nvalid) vreg[n] = *(const uint4 *)(p.v + (row0 + l * rstride) * DV + cv * VE);
    }
    // Gates: wave-wide inclusive prefix sum of clamped log alpha in fp64
    // (padding tokens: alpha = 1, beta = 0).
    if (w == 0) {
        float a = 1.f, be = 0.f;
        if (l < nvalid) {
            a = p.alpha[row0 + l * rstride];
            be = p.beta[row0 + l * rstride];
        }
        float la = logf(a);
        la = (la < kLogAlphaMin) ? kLogAlphaMin : la;  // keeps NaN
        double g = (double)la;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const double o = __shfl_up(g, d);
            if (l >= d) g += o;
        }
        sg[l] = g;
        sb[l] = be;
        sw[l] = be * expf((float)g);
        p.g[cidx * kChunk + l] = g;
    }
    // K into LDS row-major and transposed (lane = token row; padded rows are zero).
#pragma unroll
    for (int n = 0; n < DK / VE / 4; ++n) {
        const int cv = w + 4 * n;
        uint4 val = make_uint4(0u, 0u, 0u, 0u);
        if (l < nvalid) val = *(const uint4 *)(p.k + (row0 + l * rstride) * DK + cv * VE);
        *(uint4 *)(sK + l * L::LDK + cv * VE) = val;
        const E *e = (const E *)&val;
#pragma unroll
        for (int u = 0; u < VE; ++u) sKt[(cv * VE + u) * L::LDT + l] = e[u];
    }
    // Upper block-triangle of T is zero.
    for (int idx = tid; idx < kChunk * kChunk; idx += 256) {
        const int r = idx >> 6, s2 = idx & 63;
        if ((s2 >> 4) > (r >> 4)) sT[r * L::LDA + s2] = 0.f;
    }
    lds_barrier();
    if (w == 0) sd[l] = expf((float)(sg[kChunk - 1] - sg[l]));

    // A = strict_lower(beta_r e^{g_r - g_s} K K^T): the 10 lower 16x16 blocks.
    for (int t = w; t < 10; t += 4) {
        const int bi = (t >= 6) ? 3 : (t >= 3) ? 2 : (t >= 1) ? 1 : 0;
        const int bj = t - bi * (bi + 1) / 2;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < DK / 32; ++kb) {
            auto fa = load_frag<E>(sK + (16 * bi + li) * L::LDK + 32 * kb, lg);
            auto fb = load_frag<E>(sK + (16 * bj + li) * L::LDK + 32 * kb, lg);
            acc = TR::mma(fa, fb, acc);
        }
        const int s2 = 16 * bj + li;
        const double gs = sg[s2];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int r = 16 * bi + 4 * lg + q;
            float val = 0.f;
            if (s2 < r) val = sb[r] * expf((float)(sg[r] - gs)) * acc[q];
            sA[r * L::LDA + s2] = val;
        }
    }
    lds_barrier();

    // T = (I + A)^{-1}, fp32.  Diagonal 16x16 blocks by forward substitution,
    // one block per wave, one column per lane.
    if (l < 16) {
        const int base = 16 * w, j = l;
        float x[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float acc = (r == j) ? 1.f : 0.f;
#pragma unroll
            for (int s2 = 0; s2 < r; ++s2) acc -= sA[(base + r) * L::LDA + base + s2] * x[s2];
            x[r] = acc;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) sT[(base + r) * L::LDA + base + j] = x[r];
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
    // A is dead: V^T takes its place.
#pragma unroll
    for (int n = 0; n < NVV; ++n) {
        const int cv = w + 4 * n;
        const E *e = (const E *)&vreg[n];
#pragma unroll
        for (int u = 0; u < VE; ++u) sVt[(cv * VE + u) * L::LDT + l] = e[u];
    }

    // A operands of W = T diag(beta e^g) K and Ut = T diag(beta) V.
    typename TR::frag aw[4][2], au[4][2];
#pragma unroll
    for (int bi = 0; bi < 4; ++bi) {
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            const int s0 = 32 * m + 8 * lg, s1 = s0 + 4;
            const float *trow = sT + (16 * bi + li) * L::LDA + s0;
            const f32x4 tlo = *(const f32x4 *)trow;
            const f32x4 thi = *(const f32x4 *)(trow + 4);
            f32x4 wl, wh, ul, uh;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                wl[q] = tlo[q] * sw[s0 + q];
                wh[q] = thi[q] * sw[s1 + q];
                ul[q] = tlo[q] * sb[s0 + q];
                uh[q] = thi[q] * sb[s1 + q];
            }
            aw[bi][m] = TR::cat(TR::from_f32(wl), TR::from_f32(wh));
            au[bi][m] = TR::cat(TR::from_f32(ul), TR::from_f32(uh));
        }
    }
    // W tiles, staged in LDS over the dead K buffer.
    E *sW = sK;
    for (int dt = w; dt < DK / 16; dt += 4) {
        auto b0 = load_frag<E>(sKt + (16 * dt + li) * L::LDT, lg);
        auto b1 = load_frag<E>(sKt + (16 * dt + li) * L::LDT + 32, lg);
#pragma unroll
        for (int bi = 0; bi < 4; ++bi) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            acc = TR::mma(aw[bi][0], b0, acc);
            if (bi >= 2) acc = TR::mma(aw[bi][1], b1, acc);
            const auto qv = TR::from_f32(acc);
            const E *e = (const E *)&qv;
#pragma unroll
            for (int q = 0; q < 4; ++q) sW[(16 * bi + 4 * lg + q) * L::LDK + 16 * dt + li] = e[q];
        }
    }
    // Kt = (diag(e^{g_C - g}) K)^T, token-contiguous rows.
    E *Kt = p.Kt + cidx * (size_t)DK * kChunk;
    for (int idx = tid; idx < DK * (kChunk / 4); idx += 256) {
        const int d = idx >> 4, s2 = (idx & 15) * 4;
        const f32x4 kv = TR::to_f32(TR::load(sKt + d * L::LDT + s2));
        f32x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = kv[q] * sd[s2 + q];
        TR::store(Kt + d * kChunk + s2, TR::from_f32(o));
    }
    lds_barrier();
    // Ut tiles, written straight out transposed (4 consecutive tokens per lane).
    E *Ut = p.Ut + cidx * (size_t)DV * kChunk;
    for (int jt = w; jt < DV / 16; jt += 4) {
        auto b0 = load_frag<E>(sVt + (16 * jt + li) * L::LDT, lg);
        auto b1 = load_frag<E>(sVt + (16 * jt + li) * L::LDT + 32, lg);
#pragma unroll
        for (int bi = 0; bi < 4; ++bi) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            acc = TR::mma(au[bi][0], b0, acc);
            if (bi >= 2) acc = TR::mma(au[bi][1], b1, acc);
            TR::store(Ut + (16 * jt + li) * kChunk + 16 * bi + 4 * lg, TR::from_f32(acc));
        }
    }
    // W staging -> global, 16-byte coalesced.
    {
        E *Wg = p.W + cidx * (size_t)kChunk * DK;
        for (int idx = tid; idx < kChunk * (DK / VE); idx += 256) {
            const int r = idx / (DK / VE), cv = idx - r * (DK / VE);
            *(uint4 *)(Wg + r * DK + cv * VE) = *(const uint4 *)(sW + r * L::LDK + cv * VE);
        }
    }
}

// --------------------------------------------------------------------------
// Stage 2: sequential state scan across chunks.  1-D grid of
// (Dv/16) * 8 * ceil(B*H / 8) workgroups; one workgroup owns 16 state columns
// of one (b, h) and carries them through all
// chunks in fp32 accumulators.  Its DK/32 waves split the Dk rows (32 each),
// so every chunk costs one cross-wave reduction of the partial W H products.
// --------------------------------------------------------------------------
template <class E, int DK, int DV>
__global__ __launch_bounds__(DK * 2) __attribute__((amdgpu_waves_per_eu(1, 1)))
void gdn_scan_kernel(Params<E> p) {
    using TR = Tr<E>;
    using frag = typename TR::frag;
    using quad = typename TR::quad;
    constexpr int NW = DK / 32;        // waves; wave w owns state rows [32w, 32w+32)
    constexpr int NOWN = 4 / NW;       // token tiles each wave reduces
    constexpr int PF = sizeof(E) == 2 ? 4 : 2;  // chunks of operands kept in flight
    __shared__ f32x4 sP[NW][4][64];    // partial (W H) tiles
    __shared__ quad sU[4][64];         // U tiles, already rounded to E

    // XCD-aware placement: workgroups are dealt round-robin to the 8 XCDs, so
    // id = 8 slot + x runs on XCD x.  The NJ column blocks of one (b, h) are
    // given consecutive slots of the same XCD and share its L2 for the
    // chunk operands W and Kt that all of them read.
    constexpr int NJ = DV / 16;
    const int id = blockIdx.x, x = id & 7, slot = id >> 3;
    const int bh = (slot / NJ) * 8 + x, jt = slot % NJ;
    if (bh >= p.B * p.H) return;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lg = l >> 4;
    const int j0 = 16 * jt, d0 = 32 * w;
    const int j = j0 + li;  // this lane's state column

    // H rows d0 + [0, 32) as two accumulator tiles in P32 order:
    // Hacc[a][q] = H[d0 + 8 lg + 4 a + q][j].
    f32x4 Hacc[2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            Hacc[a][q] = p.state_in
                             ? p.state_in[((size_t)bh * DK + d0 + 8 * lg + 4 * a + q) * DV + j]
                             : 0.f;

    // Token tile st = 2 m + a of a chunk is produced in P32 order inside the
    // 32-token block m: its tile row i is token 32 m + p32_row(a, i).
    struct Pre {
        frag wf[4];      // A operand: W[32 m + p32_row(a, li)][d0 + k]
        frag kf[2][2];   // A operand: Kt[d0 + p32_row(a, li)][32 m + k]
        quad uq[NOWN];   // Ut^T[j][32 m + 8 lg + 4 a + q] of the owned token tiles
        double gC;       // g at the chunk's last token
    };
    auto fetch = [&](int c, Pre &f) {
        const size_t cidx = (size_t)bh * p.NC + c;
        const E *Wc = p.W + cidx * (size_t)kChunk * DK;
        const E *Kc = p.Kt + cidx * (size_t)DK * kChunk;
        const E *Uc = p.Ut + cidx * (size_t)DV * kChunk + (size_t)j * kChunk + 8 * lg;
#pragma unroll
        for (int st = 0; st < 4; ++st)
            f.wf[st] = load_frag<E>(Wc + (32 * (st >> 1) + p32_row(st & 1, li)) * DK + d0, lg);
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int m = 0; m < 2; ++m)
                f.kf[a][m] = load_frag<E>(Kc + (d0 + p32_row(a, li)) * kChunk + 32 * m, lg);
#pragma unroll
        for (int o = 0; o < NOWN; ++o) {
            const int st = w + NW * o;
            f.uq[o] = TR::load(Uc + 32 * (st >> 1) + 4 * (st & 1));
        }
        f.gC = p.g[cidx * kChunk + kChunk - 1];
        // Keep the whole fetch group together: a load scheduled into a later step
        // looks younger than the next slots' loads and forces an early full wait.
        __builtin_amdgcn_sched_barrier(0);
    };
    auto step = [&](int c, const Pre &f) {
        const size_t cidx = (size_t)bh * p.NC + c;
        // H_{c-1} rounded to E: B operand over this wave's 32 rows, and saved for stage 3.
        const frag hb = TR::cat(TR::from_f32(Hacc[0]), TR::from_f32(Hacc[1]));
        TR::store8(p.Hs + cidx * (size_t)DV * DK + (size_t)j * DK + d0 + 8 * lg, hb);
        // Partial W H over this wave's rows: four independent MFMAs, then the LDS exchange.
        f32x4 part[4];
#pragma unroll
        for (int st = 0; st < 4; ++st) part[st] = TR::mma(f.wf[st], hb, f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
        for (int st = 0; st < 4; ++st) sP[w][st][l] = part[st];
        lds_barrier();
        E *Us = p.Us + cidx * (size_t)DV * kChunk + (size_t)j * kChunk + 8 * lg;
#pragma unroll
        for (int o = 0; o < NOWN; ++o) {
            const int st = w + NW * o;
            f32x4 pr[NW];
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) pr[ww] = sP[ww][st][l];
            f32x4 u = TR::to_f32(f.uq[o]);
#pragma unroll
            for (int ww = 0; ww < NW; ++ww) u -= pr[ww];
            const quad uqr = TR::from_f32(u);
            TR::store(Us + 32 * (st >> 1) + 4 * (st & 1), uqr);
            sU[st][l] = uqr;
        }
        lds_barrier();
        const frag u0 = TR::cat(sU[0][l], sU[1][l]);
        const frag u1 = TR::cat(sU[2][l], sU[3][l]);
        const float gam = expf((float)f.gC);
#pragma unroll
        for (int a = 0; a < 2; ++a) {
            Hacc[a] *= gam;
            Hacc[a] = TR::mma(f.kf[a][0], u0, Hacc[a]);
            Hacc[a] = TR::mma(f.kf[a][1], u1, Hacc[a]);
        }
    };

    // Operands for chunk c live in ring slot c % PF and are fetched PF chunks
    // ahead.  The main loop is branch-free (fetches past the end re-read the
    // last chunk and are never used) so the compiler can keep every slot's
    // loads in flight across iterations.
    Pre ring[PF];
#pragma unroll
    for (int i = 0; i < PF; ++i) fetch(min(i, p.NC - 1), ring[i]);
    int c0 = 0;
    for (; c0 + PF <= p.NC; c0 += PF) {
#pragma unroll
        for (int i = 0; i < PF; ++i) {
            step(c0 + i, ring[i]);
            fetch(min(c0 + i + PF, p.NC - 1), ring[i]);
        }
    }
#pragma unroll
    for (int i = 0; i < PF; ++i)
        if (c0 + i < p.NC) step(c0 + i, ring[i]);

    if (p.state_out) {
#pragma unroll
        for (int a = 0; a < 2; ++a)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                p.state_out[((size_t)bh * DK + d0 + 8 * lg + 4 * a + q) * DV + j] = Hacc[a][q];
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

    stage_rows<E, DK, 256>(sH, L::LDH, p.Hs + cidx * (size_t)DV * DK, DK, DV, DV, tid);
    stage_rows<E, kChunk, 256>(sU, L::LDU, p.Us + cidx * (size_t)DV * kChunk, kChunk, DV, DV, tid);
    stage_rows<E, DK, 256>(sK, L::LDK, p.k + row0 * DK, rstride * DK, kChunk, nvalid, tid);
    if (tid < kChunk) sg[tid] = p.g[cidx * kChunk + tid];

    // Q rows of this wave's tokens as B operands (B[k=d][n=r] = Q[r][d]); padded tokens are 0.
    const int r = 16 * w + li;  // token within the chunk
    const bool rvalid = r < nvalid;
    frag qf[DK / 32];
#pragma unroll
    for (int kb = 0; kb < DK / 32; ++kb) {
        if (rvalid) {
            qf[kb] = load_frag<E>(p.q + (row0 + r * rstride) * DK + 32 * kb, lg);
        } else {
            qf[kb] = TR::cat(TR::zero(), TR::zero());
        }
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

    E *orow = p.out + (row0 + r * rstride) * DV;
#pragma unroll 2
    for (int jt = 0; jt < DV / 16; ++jt) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < DK / 32; ++kb)
            acc = TR::mma(load_frag<E>(sH + (16 * jt + li) * L::LDH + 32 * kb, lg), qf[kb], acc);
        acc *= er;
        acc = TR::mma(load_frag<E>(sU + (16 * jt + li) * L::LDU, lg), pf0, acc);
        if (w >= 2) acc = TR::mma(load_frag<E>(sU + (16 * jt + li) * L::LDU + 32, lg), pf1, acc);
        if (rvalid) TR::store(orow + 16 * jt + 4 * lg, TR::from_f32(acc));
    }
}

}  // namespace gdn
