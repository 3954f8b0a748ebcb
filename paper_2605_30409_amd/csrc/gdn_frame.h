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
//   gdn_frame_summary_kernel  (token split s, half c, frame f, head): the
//       half c = 0 accumulates G, c = 1 accumulates A, over the split's
//       tokens (64-token blocks staged in LDS); writes fp32 partial tiles.
//   gdn_frame_reduce_kernel   sums the NS splits' partials and applies the
//       key scale: G as ready-made MFMA operand fragments (E), A as fp32
//       accumulator tiles.
//   gdn_frame_scan_kernel     one wave per (head, 16 state columns): H_f for
//       every frame in turn, written as the output kernel's operand
//       fragments (E), and the terminal state.
//   gdn_frame_output_kernel   64 * NTW tokens of one frame per workgroup:
//       O^T = H_f^T Q^T.
//
// Tile layouts (see gdn_device.h for the lane conventions).  Accumulator
// tiles over the Dk rows are in P32 order: row tile r = 2 m + a holds rows
// 32 m + p32_row(a, i), so lane (li, lg) holds rows 32 m + 8 lg + 4 a + q.
// G tiles are in P32 order along the columns too.  Because G is symmetric,
// the pair of partial tiles (r = 2 kb, c = t), (r = 2 kb + 1, c = t) is, lane
// by lane, the A operand fragment of row tile t of G over the k block kb.
#pragma once

#include "gdn_device.h"

namespace gdn {

template <class E> struct FrameParams {
    const E *q, *k, *v;          // [B][T][H][Dk] / [Dv], T = F * N
    const float *alpha;          // [B][F][H]
    const float *beta;           // [B][T][H]
    const float *state_in;       // [B][H][Dk][Dv] or null (zero)
    E *out;                      // [B][T][H][Dv]
    float *state_out;            // [B][H][Dk][Dv] or null
    int B, H, F, N;
    int NS, NBT;                 // token splits per frame, tokens per split (a multiple of 64)
    int OB;                      // output workgroups per frame
    float key_scale;
    float *PG;                   // [B*H][F][NS][Dk/16][Dk/16][64][4]  partial G tiles
    float *PA;                   // [B*H][F][NS][Dk/16][Dv/16][64][4]  partial A tiles
    E *Gf;                       // [B*H][F][Dk/16][Dk/32][64][8]      G operand fragments
    float *Af;                   // [B*H][F][Dk/16][Dv/16][64][4]      A tiles
    E *Hf;                       // [B*H][F][Dv/16][Dk/32][64][8]      H_f operand fragments
};

// Workgroups of the summary kernel: the two halves of one (split, frame,
// head) unit get block ids 8 apart, i.e. the same XCD (blocks are dealt to the
// 8 XCDs round robin), so the keys both of them stage are read from HBM once.
inline unsigned frame_summary_blocks(long long units) { return 16u * (unsigned)((units + 7) / 8); }
// Output and scan grids: all workgroups of one unit (a (frame, head) or a
// head) on one XCD, so the state they share is fetched into one L2.
inline unsigned xcd_blocks(long long units, int per_unit) {
    return 8u * (unsigned)per_unit * (unsigned)((units + 7) / 8);
}
__device__ __forceinline__ void xcd_unit(int id, int per_unit, int &unit, int &sub) {
    const int x = id & 7, y = id >> 3;
    sub = y % per_unit;
    unit = 8 * (y / per_unit) + x;
}

template <class E, int DK, int DV> struct FrameSumLds {
    static constexpr int PAD = 16 / (int)sizeof(E);
    static constexpr int DY = DK > DV ? DK : DV;
    static constexpr int LDK = DK + PAD, LDY = DY + PAD;
    static constexpr size_t oK = 0;                              // raw keys, token rows
    static constexpr size_t oY = oK + sizeof(E) * 64 * LDK;      // beta * (keys or values)
    static constexpr size_t bytes = oY + sizeof(E) * 64 * LDY;
};

// beta times the 16 / sizeof(E) elements of a 16-byte vector, rounded to E.
template <class E> __device__ __forceinline__ u32x4 scale_vec(u32x4 x, float b);
template <> __device__ __forceinline__ u32x4 scale_vec<uint16_t>(u32x4 x, float b) {
    u32x4 y;
#pragma unroll
    for (int e = 0; e < 4; ++e) y[e] = pack_bf16x2(__uint_as_float(x[e] << 16) * b, __uint_as_float(x[e] & 0xffff0000u) * b);
    return y;
}
template <> __device__ __forceinline__ u32x4 scale_vec<float>(u32x4 x, float b) {
    return __builtin_bit_cast(u32x4, __builtin_bit_cast(f32x4, x) * b);
}

// Phase A for one half.  YV = false: C = K^T B K (Dk x Dk, P32 columns);
// YV = true: C = K^T B V (Dk x Dv).  Waves form a 2 x 2 grid over the row and
// column tiles; a lane's 16-byte vectors of the next block are loaded into
// registers while the current block is multiplied.
template <class E, int DK, int DV, bool YV>
__device__ __forceinline__ void frame_summary_half(const FrameParams<E> &p, unsigned char *smem, int s, int f,
                                                   int bh) {
    using L = FrameSumLds<E, DK, DV>;
    using TR = Tr<E>;
    using frag = typename TR::frag;
    constexpr int DY = YV ? DV : DK;
    constexpr int NR = DK / 16, NC = DY / 16, RPW = NR / 2, CPW = NC / 2;
    constexpr int VE = 16 / (int)sizeof(E);
    constexpr int KPR = DK / VE, YPR = DY / VE;               // 16-byte vectors per row
    constexpr int NKV = 64 * KPR / 256, NYV = YV ? 64 * YPR / 256 : 1;
    E *sK = (E *)(smem + L::oK), *sY = (E *)(smem + L::oY);

    const int b = bh / p.H, h = bh - b * p.H;
    const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), l = tid & 63, li = l & 15,
              lg = l >> 4;
    const int wr = w >> 1, wc = w & 1;
    const size_t T = (size_t)p.F * p.N;
    const int t_lo = f * p.N + s * p.NBT;
    const int t_hi = min(f * p.N + p.N, t_lo + p.NBT);
    const size_t row_b = (size_t)b * T;

    // One block's 16-byte vectors in registers.  Rows past the split are read
    // from its last token (always in bounds) with beta = 0: their scaled
    // copies are zero, so they add nothing.
    struct Blk {
        u32x4 k[NKV], y[NYV];
        float kb[NKV], yb[NYV];
    };
    auto load_block = [&](int t0) {
        Blk r;
#pragma unroll
        for (int j = 0; j < NKV; ++j) {
            const int i = tid + 256 * j, t = t0 + i / KPR;
            const size_t row = (row_b + min(t, t_hi - 1)) * p.H + h;
            r.k[j] = *(const u32x4 *)(p.k + row * DK + (i % KPR) * VE);
            const float be = p.beta[row];
            r.kb[j] = t < t_hi ? be : 0.f;
        }
#pragma unroll
        for (int j = 0; j < NYV; ++j) {
            r.y[j] = u32x4{0u, 0u, 0u, 0u};
            r.yb[j] = 0.f;
            if constexpr (YV) {
                const int i = tid + 256 * j, t = t0 + i / YPR;
                const size_t row = (row_b + min(t, t_hi - 1)) * p.H + h;
                r.y[j] = *(const u32x4 *)(p.v + row * DV + (i % YPR) * VE);
                const float be = p.beta[row];
                r.yb[j] = t < t_hi ? be : 0.f;
            }
        }
        return r;
    };

    f32x4 acc[RPW][CPW];
#pragma unroll
    for (int i = 0; i < RPW; ++i)
#pragma unroll
        for (int j = 0; j < CPW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    Blk cur = load_block(t_lo);
    for (int t0 = t_lo; t0 < t_hi; t0 += 64) {
#pragma unroll
        for (int j = 0; j < NKV; ++j) {
            const int i = tid + 256 * j, r = i / KPR, c = (i % KPR) * VE;
            *(u32x4 *)(sK + r * L::LDK + c) = cur.k[j];
            if (!YV) *(u32x4 *)(sY + r * L::LDY + c) = scale_vec<E>(cur.k[j], cur.kb[j]);
        }
        if constexpr (YV) {
#pragma unroll
            for (int j = 0; j < NYV; ++j) {
                const int i = tid + 256 * j;
                *(u32x4 *)(sY + (i / YPR) * L::LDY + (i % YPR) * VE) = scale_vec<E>(cur.y[j], cur.yb[j]);
            }
        }
        lds_barrier();
        if (t0 + 64 < t_hi) cur = load_block(t0 + 64);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            frag af[RPW], bf[CPW];
#pragma unroll
            for (int i = 0; i < RPW; ++i) {
                const int r = RPW * wr + i;
                af[i] = tr_frag<E>(sK, L::LDK, 32 * kb, 32 * (r >> 1), true, r & 1, li, lg);
            }
#pragma unroll
            for (int j = 0; j < CPW; ++j) {
                const int c = CPW * wc + j;
                bf[j] = YV ? tr_frag<E>(sY, L::LDY, 32 * kb, 16 * c, false, 0, li, lg)
                           : tr_frag<E>(sY, L::LDY, 32 * kb, 32 * (c >> 1), true, c & 1, li, lg);
            }
#pragma unroll
            for (int i = 0; i < RPW; ++i)
#pragma unroll
                for (int j = 0; j < CPW; ++j) acc[i][j] = TR::mma(af[i], bf[j], acc[i][j]);
        }
        lds_barrier();
    }
    float *dst = (YV ? p.PA : p.PG) + (((size_t)bh * p.F + f) * p.NS + s) * (size_t)NR * NC * 256;
#pragma unroll
    for (int i = 0; i < RPW; ++i)
#pragma unroll
        for (int j = 0; j < CPW; ++j)
            *(f32x4 *)(dst + ((size_t)((RPW * wr + i) * NC + CPW * wc + j) * 64 + l) * 4) = acc[i][j];
}

template <class E, int DK, int DV>
__global__ __launch_bounds__(256) void gdn_frame_summary_kernel(FrameParams<E> p) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int id = blockIdx.x;
    const int half = (id >> 3) & 1, u = (id & 7) + 8 * (id >> 4);
    if (u >= p.NS * p.F * p.B * p.H) return;
    const int s = u % p.NS, rest = u / p.NS, f = rest % p.F, bh = rest / p.F;
    if (half == 0)
        frame_summary_half<E, DK, DV, false>(p, smem, s, f, bh);
    else
        frame_summary_half<E, DK, DV, true>(p, smem, s, f, bh);
}

// Sum over the splits.  Items per (frame, head): the Dk/16 x Dk/32 G operand
// fragments, then the Dk/16 x Dv/16 A tiles; one wave per item.
template <class E, int DK, int DV>
__global__ __launch_bounds__(256) void gdn_frame_reduce_kernel(FrameParams<E> p) {
    using TR = Tr<E>;
    constexpr int NR = DK / 16, KB = DK / 32, NCV = DV / 16;
    constexpr int NGI = NR * KB, NI = NGI + NR * NCV;
    const int item = blockIdx.y * 4 + (threadIdx.x >> 6);
    const size_t fi = blockIdx.x;                                // (b*H + h) * F + f
    if (item >= NI) return;
    const int l = threadIdx.x & 63;
    if (item < NGI) {
        const int t = item / KB, kb = item - t * KB;
        const float *src = p.PG + fi * p.NS * (size_t)NR * NR * 256 + l * 4;
        f32x4 lo = {0.f, 0.f, 0.f, 0.f}, hi = lo;
        for (int s = 0; s < p.NS; ++s) {
            const float *ps = src + (size_t)s * NR * NR * 256;
            lo += *(const f32x4 *)(ps + (size_t)((2 * kb) * NR + t) * 256);
            hi += *(const f32x4 *)(ps + (size_t)((2 * kb + 1) * NR + t) * 256);
        }
        const float k2 = p.key_scale * p.key_scale;
        TR::store8(p.Gf + ((fi * NR + t) * KB + kb) * 512 + l * 8,
                   TR::cat(TR::from_f32(lo * k2), TR::from_f32(hi * k2)));
    } else {
        const int a = item - NGI;                                // = t * NCV + jt
        const float *src = p.PA + fi * p.NS * (size_t)NR * NCV * 256 + (size_t)a * 256 + l * 4;
        f32x4 sum = {0.f, 0.f, 0.f, 0.f};
        for (int s = 0; s < p.NS; ++s) sum += *(const f32x4 *)(src + (size_t)s * NR * NCV * 256);
        *(f32x4 *)(p.Af + (fi * NR * NCV + a) * 256 + l * 4) = sum * p.key_scale;
    }
}

// Phase B.  One wave per (head, column tile jt): Hacc[t][q] =
// H[32 (t / 2) + 8 lg + 4 (t % 2) + q][16 jt + li], carried through the frames
// in fp32.  The product G H takes H rounded to E as the B operand.
template <class E, int DK, int DV>
__global__ __launch_bounds__(64) void gdn_frame_scan_kernel(FrameParams<E> p) {
    using TR = Tr<E>;
    using frag = typename TR::frag;
    constexpr int NT = DK / 16, KB = DK / 32, NJ = DV / 16;
    int bh, jt;
    xcd_unit(blockIdx.x, NJ, bh, jt);
    if (bh >= p.B * p.H) return;
    const int b = bh / p.H, h = bh - b * p.H;
    const int l = threadIdx.x & 63, li = l & 15, lg = l >> 4;
    const int col = 16 * jt + li;
    f32x4 Hacc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int r0 = 32 * (t >> 1) + 8 * lg + 4 * (t & 1);
#pragma unroll
        for (int q = 0; q < 4; ++q)
            Hacc[t][q] = p.state_in ? p.state_in[((size_t)bh * DK + r0 + q) * DV + col] : 0.f;
    }
    for (int f = 0; f < p.F; ++f) {
        const size_t fi = (size_t)bh * p.F + f;
        const float a = p.alpha[((size_t)b * p.F + f) * p.H + h];
        const E *G = p.Gf + fi * NT * KB * 512 + l * 8;
        const float *A = p.Af + fi * NT * NJ * 256 + l * 4;
        frag hb[KB];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) hb[kb] = TR::cat(TR::from_f32(Hacc[2 * kb]), TR::from_f32(Hacc[2 * kb + 1]));
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            f32x4 gh = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) gh = TR::mma(TR::load8(G + (t * KB + kb) * 512), hb[kb], gh);
            const f32x4 av = *(const f32x4 *)(A + (t * NJ + jt) * 256);
            Hacc[t] = a * (Hacc[t] - gh) + av;
        }
        E *hf = p.Hf + (fi * NJ + jt) * (size_t)KB * 512 + l * 8;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
            TR::store8(hf + kb * 512, TR::cat(TR::from_f32(Hacc[2 * kb]), TR::from_f32(Hacc[2 * kb + 1])));
    }
    if (p.state_out) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int r0 = 32 * (t >> 1) + 8 * lg + 4 * (t & 1);
#pragma unroll
            for (int q = 0; q < 4; ++q) p.state_out[((size_t)bh * DK + r0 + q) * DV + col] = Hacc[t][q];
        }
    }
}

// Phase C.  A workgroup takes 64 NTW tokens of one frame; wave w the 16 NTW
// tokens from 16 NTW w.  H_f's fragments are staged in LDS once per
// workgroup.  Lane (li, lg) of fragment (jo, kb) holds H_f[32 kb + 8 lg + q'][16 jo + li]:
// the A operand of row 16 jo + li of H_f^T.  With the query rows as B operand
// the product tile is O^T, and lane (li, lg) gets O[token li][16 jo + 4 lg + q].
template <class E> struct FrameOutNTW { static constexpr int value = sizeof(E) == 2 ? 4 : 2; };

template <class E, int DK, int DV> struct FrameOutLds {
    static constexpr size_t bytes = sizeof(E) * DK * DV;
};

template <class E, int DK, int DV>
__global__ __launch_bounds__(256) void gdn_frame_output_kernel(FrameParams<E> p) {
    using TR = Tr<E>;
    using frag = typename TR::frag;
    constexpr int KB = DK / 32, NJ = DV / 16, NTW = FrameOutNTW<E>::value;
    constexpr int HV = DV * DK * (int)sizeof(E) / 16;         // 16-byte vectors of H_f
    static_assert(HV % 256 == 0, "whole vectors per thread");
    extern __shared__ __align__(16) unsigned char smem[];
    int unit, blk;
    xcd_unit(blockIdx.x, p.OB, unit, blk);
    if (unit >= p.F * p.B * p.H) return;
    const int bh = unit / p.F, f = unit - bh * p.F;
    const int b = bh / p.H, h = bh - b * p.H;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lg = l >> 4;
    const size_t fi = (size_t)bh * p.F + f;

    const u32x4 *src = (const u32x4 *)(p.Hf + fi * (size_t)DV * DK);
#pragma unroll
    for (int j = 0; j < HV / 256; ++j) ((u32x4 *)smem)[tid + 256 * j] = src[tid + 256 * j];

    const size_t T = (size_t)p.F * p.N;
    const int n0 = 64 * NTW * blk + 16 * NTW * w;
    frag qf[NTW][KB];
#pragma unroll
    for (int i = 0; i < NTW; ++i) {
        const int n = min(n0 + 16 * i + li, p.N - 1);
        const E *qrow = p.q + (((size_t)b * T + (size_t)f * p.N + n) * p.H + h) * DK;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) qf[i][kb] = load_frag<E>(qrow + 32 * kb, lg);
    }
    lds_barrier();
    const E *sH = (const E *)smem + l * 8;
#pragma unroll
    for (int jo = 0; jo < NJ; ++jo) {
        frag hfr[KB];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) hfr[kb] = TR::load8(sH + (jo * KB + kb) * 512);
#pragma unroll
        for (int i = 0; i < NTW; ++i) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) acc = TR::mma(hfr[kb], qf[i][kb], acc);
            const int n = n0 + 16 * i + li;
            if (n < p.N)
                TR::store(p.out + (((size_t)b * T + (size_t)f * p.N + n) * p.H + h) * DV + 16 * jo + 4 * lg,
                          TR::from_f32(acc));
        }
    }
}

}  // namespace gdn
