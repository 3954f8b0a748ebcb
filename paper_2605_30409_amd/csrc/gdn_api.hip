// Host side of libgdn: argument validation, workspace layout and caching,
// kernel launches, and the extern "C" entry points declared in gdn.h.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <unordered_map>
#include <vector>

#include "gdn.h"
#include "gdn_frame.h"
#include "gdn_kernels.h"

namespace {

using gdn::kChunk;
using gdn::kGateRec;

struct WsLayout {
    size_t g, gf, W, Ut, Hs, Us, Nf, PsiT, lgam, HgT, total;
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int num_chunks(int T) { return (T + kChunk - 1) / kChunk; }

// Chunks per scan group.  bf16: a single group (one sequential scan per
// (b, h) with the output fused into it) whenever the (b, h) streams give at
// least 64 column-tile workgroups -- measured faster than any grouped scan on
// the 3-frame, batched and 12-frame workloads -- or the sequence has at most 64
// chunks.  fp32, and bf16 with fewer streams: a single group when the sequence
// is short or when the streams alone fill the chip; otherwise about sqrt(NC)
// chunks per group, which balances the group-parallel passes (two passes over
// G chunks) against the sequential scan over NC / G groups.
int auto_group(int NC, long long BH, int Dv, bool bf16) {
    if (NC <= 64 || BH * (Dv / 16) >= (bf16 ? 64 : 512)) return NC;
    int G = (int)(__builtin_sqrt((double)NC) + 0.5);
    return G < 2 ? 2 : G;
}

int resolve_group(int NC, long long BH, int Dv, int group, bool bf16) {
    if (group <= 0) group = auto_group(NC, BH, Dv, bf16);
    return group > NC ? NC : group;
}

WsLayout ws_layout(int B, int H, int T, int Dk, int Dv, size_t esz, int G) {
    const int NC = num_chunks(T);
    const int NG = (NC + G - 1) / G;
    const size_t bh = (size_t)B * H;
    const size_t nch = bh * NC;
    const size_t ngr = NG > 1 ? bh * NG : 0;
    WsLayout L;
    size_t off = 0;
    L.g = off;    off = align256(off + nch * kChunk * 8);
    L.gf = off;   off = align256(off + nch * kGateRec * 4);
    L.W = off;    off = align256(off + nch * kChunk * Dk * esz);
    L.Ut = off;   off = align256(off + nch * Dv * kChunk * esz);
    // With the output fused into the scan (bf16, one group) these regions hold
    // the chunk's decay-scaled queries (C x Dk) and masked scores (C x C)
    // instead of the per-chunk state (Dv x Dk) and pseudo-values (Dv x C).
    const bool fused = esz == 2 && NG == 1;
    L.Hs = off;   off = align256(off + nch * (fused ? kChunk : Dv) * Dk * esz);
    L.Us = off;   off = align256(off + nch * (fused ? kChunk : Dv) * kChunk * esz);
    L.Nf = off;   off = align256(off + ngr * Dk * Dk * esz);
    L.PsiT = off; off = align256(off + ngr * Dv * Dk * 4);
    L.lgam = off; off = align256(off + ngr * 8);
    L.HgT = off;  off = align256(off + ngr * Dv * Dk * 4);
    L.total = off;
    return L;
}

// Bytes each workspace region must span for the kernels that use it, from the
// kernels' index expressions evaluated at their largest indices (chunk index
// cidx = B H NC - 1, group index gidx = B H NG - 1, lane 63, last fragment):
// the highest element offset touched, plus the element's width.  0 if no
// kernel of the path uses the region.
struct WsNeeds {
    size_t g, gf, W, Ut, Hs, Us, Nf, PsiT, lgam, HgT;
};

WsNeeds ws_needs(int B, int H, int T, int Dk, int Dv, size_t esz, int G) {
    const size_t NC = (size_t)num_chunks(T), NG = (NC + G - 1) / G;
    const size_t cmax = (size_t)B * H * NC - 1;             // last chunk record
    const size_t gmax = (size_t)B * H * NG - 1;             // last group record
    const bool fused = esz == 2 && NG == 1;
    const size_t KB = (size_t)Dk / 32, NJ = (size_t)Dv / 16;
    WsNeeds n{};
    // WY kernel: g[cidx * 64 + l], gf[cidx * 68 + l] and the fp64 g_C at
    // gf + cidx * 68 + 64 (the scan copies gf[cidx * 68 + 4 l .. + 3], l < 17)
    n.g = (cmax * kChunk + 63 + 1) * 8;
    n.gf = (cmax * kGateRec + kGateRec) * 4;
    // -W fragment ((wv * 4 + st) * 2 + kb) * 512 + l * 8, 8 elements
    n.W = (cmax * kChunk * Dk + ((((size_t)Dk / 64 - 1) * 4 + 3) * 2 + 1) * 512 + 63 * 8 + 8) * esz;
    // U~t quad (4 jt + st) * 256 + l * 4, 4 elements
    n.Ut = (cmax * Dv * kChunk + (4 * (NJ - 1) + 3) * 256 + 63 * 4 + 4) * esz;
    if (fused) {
        // WY: Qf (rt * KB + kb) * 512 + l * 8 and Pf (rt * 2 + m) * 512 + l * 8
        n.Hs = (cmax * kChunk * Dk + (3 * KB + KB - 1) * 512 + 63 * 8 + 8) * esz;
        n.Us = (cmax * kChunk * kChunk + (3 * 2 + 1) * 512 + 63 * 8 + 8) * esz;
    } else {
        // chunk states: Hs[(column) * Dk + 32 kb + 8 lg], Us[(column) * 64 + 32 + 8 lg]
        n.Hs = (cmax * Dv * Dk + (size_t)(Dv - 1) * Dk + 32 * (KB - 1) + 24 + 8) * esz;
        n.Us = (cmax * Dv * kChunk + (size_t)(Dv - 1) * kChunk + 32 + 24 + 8) * esz;
    }
    if (NG > 1) {
        // group transfer: N fragments ((v * 4 + t) * (Dk / 32) + kb) * 512 + l * 8,
        // Psi^T[(gidx * Dv + column) * Dk + row], log Gamma[gidx]; group scan: H^T like Psi^T
        n.Nf = (gmax * Dk * Dk + ((((size_t)Dk / 64 - 1) * 4 + 3) * KB + KB - 1) * 512 + 63 * 8 + 8) * esz;
        n.PsiT = ((gmax * Dv + Dv - 1) * Dk + Dk) * 4;
        n.lgam = (gmax + 1) * 8;
        n.HgT = ((gmax * Dv + Dv - 1) * Dk + Dk) * 4;
    }
    return n;
}

bool shape_ok(int B, int H, int T) {
    if (B < 1 || H < 1 || T < 1) return false;
    // gridDim.y carries B*H
    if ((long long)B * H > 65535) return false;
    return true;
}

bool dims_ok(int Dk, int Dv, int chunk) {
    return (Dk == 64 || Dk == 128) && (Dv == 64 || Dv == 128) && chunk == kChunk;
}

bool misaligned(const void *p) { return p && ((uintptr_t)p & 15u); }

struct Range {
    uintptr_t lo, hi;
    bool valid() const { return lo != 0; }
    bool overlaps(const Range &o) const { return valid() && o.valid() && lo < o.hi && o.lo < hi; }
};
Range range(const void *p, size_t bytes) { return Range{(uintptr_t)p, (uintptr_t)p + bytes}; }

int validate(const void *q, const void *k, const void *v, const float *alpha, const float *beta,
             const float *state_in, const void *out, const float *state_out, int B, int H, int T,
             int Dk, int Dv, int chunk, size_t esz) {
    if (!q || !k || !v || !alpha || !beta || !out) return GDN_ERR_NULL;
    if (!shape_ok(B, H, T)) return GDN_ERR_SHAPE;
    if (!dims_ok(Dk, Dv, chunk)) return GDN_ERR_UNSUPPORTED;
    if (misaligned(q) || misaligned(k) || misaligned(v) || misaligned(alpha) || misaligned(beta) ||
        misaligned(state_in) || misaligned(out) || misaligned(state_out))
        return GDN_ERR_ALIGN;
    const size_t ntok = (size_t)B * T * H;
    const Range rq = range(q, ntok * Dk * esz), rk = range(k, ntok * Dk * esz),
                rv = range(v, ntok * Dv * esz), ra = range(alpha, ntok * 4), rb = range(beta, ntok * 4),
                ro = range(out, ntok * Dv * esz);
    const size_t sbytes = (size_t)B * H * Dk * Dv * 4;
    const Range rsi = range(state_in, sbytes), rso = range(state_out, sbytes);
    const Range ins[] = {rq, rk, rv, ra, rb, rsi};
    for (const Range &r : ins)
        if (ro.overlaps(r)) return GDN_ERR_ALIAS;
    if (rso.valid()) {
        for (int i = 0; i < 5; ++i)
            if (rso.overlaps(ins[i])) return GDN_ERR_ALIAS;
        if (rso.overlaps(ro)) return GDN_ERR_ALIAS;
        if (rsi.valid() && rso.overlaps(rsi) && rso.lo != rsi.lo) return GDN_ERR_ALIAS;
    }
    return GDN_OK;
}

template <class E>
gdn::Params<E> make_params(const void *q, const void *k, const void *v, const float *alpha,
                           const float *beta, const float *state_in, void *out, float *state_out,
                           int B, int H, int T, int Dk, int Dv, int G, void *ws) {
    gdn::Params<E> p;
    p.q = (const E *)q;
    p.k = (const E *)k;
    p.v = (const E *)v;
    p.alpha = alpha;
    p.beta = beta;
    p.state_in = state_in;
    p.out = (E *)out;
    p.state_out = state_out;
    p.B = B;
    p.H = H;
    p.T = T;
    p.NC = num_chunks(T);
    p.G = G;
    p.NG = (p.NC + G - 1) / G;
    const WsLayout L = ws_layout(B, H, T, Dk, Dv, sizeof(E), G);
    unsigned char *base = (unsigned char *)ws;
    p.g = (double *)(base + L.g);
    p.gf = (float *)(base + L.gf);
    p.W = (E *)(base + L.W);
    p.Ut = (E *)(base + L.Ut);
    p.Hs = (E *)(base + L.Hs);
    p.Us = (E *)(base + L.Us);
    // The output is fused into the scan on the bf16 path with one scan group;
    // its Q and P fragments then live in the (unused) Hs and Us regions.
    p.fused = (sizeof(E) == 2 && p.NG == 1) ? 1 : 0;
    p.Qf = p.Hs;
    p.Pf = p.Us;
    p.Nf = (E *)(base + L.Nf);
    p.PsiT = (float *)(base + L.PsiT);
    p.lgam = (double *)(base + L.lgam);
    p.HgT = (float *)(base + L.HgT);
    return p;
}

// Launch one kernel whose only argument is a parameter struct; returns the
// launch's own status (the thread's pending HIP error is neither read nor
// cleared, so an error the caller left pending is not reported as this call's).
template <class P>
hipError_t launch(const void *fn, dim3 grid, dim3 block, size_t lds, hipStream_t s, const P &p) {
    P copy = p;
    void *args[] = {&copy};
    return hipLaunchKernel(fn, grid, block, args, lds, s);
}

// The scan kernel with the output fused (bf16 only; nullptr for fp32).
template <class E, int DK, int DV> const void *fused_scan_fn() {
    if constexpr (sizeof(E) == 2)
        return (const void *)gdn::gdn_chunkscan_kernel<E, DK, DV, gdn::SCAN_STATES, 1, 1, true>;
    else
        return nullptr;
}

constexpr int kStages = 5;  // WY transform, group transfers, group scan, chunk states, output

// Stage timing (measurement aid): every stage that launches is enqueued `reps`
// times back to back between the events ev[2 s] and ev[2 s + 1].
struct StageTiming {
    int reps;
    hipEvent_t ev[2 * kStages];
    bool ran[kStages];
};

template <class E, int DK, int DV>
hipError_t launch_path(const gdn::Params<E> &p, hipStream_t s, StageTiming *tm) {
    constexpr int CT = gdn::ScanCT<E>::value;
    constexpr int NCW = gdn::kScanNCW;
    using LT = gdn::ScanLds<E, DK, CT, NCW>;  // grouped passes
    using L1 = gdn::ScanLds<E, DK, 1, 1>;     // single-group scan
    using LF = gdn::ScanLds<E, DK, 1, 1, sizeof(E) == 2>;  // single-group scan with the output fused
    constexpr unsigned scan_threads = (NCW + 2) * 64, scan_threads1 = 3 * 64, scan_threadsF = 4 * 64;
    static std::once_flag attr_once;
    static hipError_t attr_err = hipSuccess;
    const size_t lds1 = gdn::WyLds<E, DK, DV>::bytes;
    const size_t lds3 = gdn::OutLds<E, DK, DV>::bytes;
    std::call_once(attr_once, [&] {
        const struct {
            const void *fn;
            size_t bytes;
        } dyn[] = {
            {(const void *)gdn::gdn_wy_kernel<E, DK, DV>, lds1},
            {(const void *)gdn::gdn_output_kernel<E, DK, DV>, lds3},
            {(const void *)gdn::gdn_chunkscan_kernel<E, DK, DV, gdn::SCAN_TRANS, CT, NCW>, LT::bytes},
            {(const void *)gdn::gdn_chunkscan_kernel<E, DK, DV, gdn::SCAN_STATES, CT, NCW>, LT::bytes},
            {(const void *)gdn::gdn_chunkscan_kernel<E, DK, DV, gdn::SCAN_STATES, 1, 1>, L1::bytes},
            {fused_scan_fn<E, DK, DV>(), LF::bytes},
        };
        for (const auto &d : dyn) {
            if (!d.fn) continue;
            const hipError_t e =
                hipFuncSetAttribute(d.fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)d.bytes);
            if (e != hipSuccess && attr_err == hipSuccess) attr_err = e;
        }
    });
    if (attr_err != hipSuccess) return attr_err;
    const unsigned BH = (unsigned)(p.B * p.H);
    // workgroup counts: column blocks x 8 x ceil(units / 8) (see the XCD placement)
    auto groups = [](unsigned nblocks, unsigned units) { return nblocks * 8u * ((units + 7u) / 8u); };
    auto stage = [&](int i) -> hipError_t {
        switch (i) {
        case 0:
            return launch((const void *)gdn::gdn_wy_kernel<E, DK, DV>, dim3(p.NC, BH), dim3(64 * gdn::kWyWaves),
                          lds1, s, p);
        case 1:
            return launch((const void *)gdn::gdn_chunkscan_kernel<E, DK, DV, gdn::SCAN_TRANS, CT, NCW>,
                          dim3(groups((DK + DV) / (16 * CT * NCW), BH * p.NG)), dim3(scan_threads), LT::bytes, s,
                          p);
        case 2:
            return launch((const void *)gdn::gdn_groupscan_kernel<E, DK, DV>, dim3(groups(DV / 16, BH)), dim3(DK),
                          0, s, p);
        case 3:
            if (p.NG > 1)
                return launch((const void *)gdn::gdn_chunkscan_kernel<E, DK, DV, gdn::SCAN_STATES, CT, NCW>,
                              dim3(groups(DV / (16 * CT * NCW), BH * p.NG)), dim3(scan_threads), LT::bytes, s, p);
            // one sequential scan per (b, h), one column tile per workgroup,
            // which also computes the output of its columns (bf16)
            if (p.fused)
                return launch(fused_scan_fn<E, DK, DV>(), dim3(groups(DV / 16, BH)), dim3(scan_threadsF), LF::bytes,
                              s, p);
            // one sequential scan per (b, h): one column tile per compute wave
            return launch((const void *)gdn::gdn_chunkscan_kernel<E, DK, DV, gdn::SCAN_STATES, 1, 1>,
                          dim3(groups(DV / 16, BH)), dim3(scan_threads1), L1::bytes, s, p);
        default:
            return launch((const void *)gdn::gdn_output_kernel<E, DK, DV>, dim3(p.NC, BH), dim3(256), lds3, s, p);
        }
    };
    hipError_t er = hipSuccess;
    for (int i = 0; i < kStages && er == hipSuccess; ++i) {
        const bool runs = (i == 1 || i == 2) ? p.NG > 1 : (i == 4 ? !p.fused : true);
        if (tm) tm->ran[i] = runs;
        if (!runs) continue;
        if (!tm) {
            er = stage(i);
            continue;
        }
        er = hipEventRecord(tm->ev[2 * i], s);
        for (int r = 0; r < tm->reps && er == hipSuccess; ++r) er = stage(i);
        if (er == hipSuccess) er = hipEventRecord(tm->ev[2 * i + 1], s);
    }
    return er;
}

template <class E>
hipError_t dispatch(const gdn::Params<E> &p, int Dk, int Dv, hipStream_t s, StageTiming *tm) {
    if (Dk == 128 && Dv == 128) return launch_path<E, 128, 128>(p, s, tm);
    if (Dk == 64 && Dv == 64) return launch_path<E, 64, 64>(p, s, tm);
    if (Dk == 128 && Dv == 64) return launch_path<E, 128, 64>(p, s, tm);
    return launch_path<E, 64, 128>(p, s, tm);
}

int run(const void *q, const void *k, const void *v, const float *alpha, const float *beta,
        const float *state_in, void *out, float *state_out, int B, int H, int T, int Dk, int Dv,
        int chunk, bool bf16, int group, void *ws, size_t ws_bytes, void *stream, StageTiming *tm) {
    const size_t esz = bf16 ? 2 : 4;
    int st = validate(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, esz);
    if (st != GDN_OK) return st;
    const int G = resolve_group(num_chunks(T), (long long)B * H, Dv, group, bf16);
    if (!ws || ((uintptr_t)ws & 255u) || ws_bytes < ws_layout(B, H, T, Dk, Dv, esz, G).total)
        return GDN_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (bf16) {
        e = dispatch(make_params<uint16_t>(q, k, v, alpha, beta, state_in, out, state_out, B, H, T,
                                           Dk, Dv, G, ws),
                     Dk, Dv, s, tm);
    } else {
        e = dispatch(make_params<float>(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk,
                                        Dv, G, ws),
                     Dk, Dv, s, tm);
    }
    return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

// Library-cached workspace, one buffer per device, grown on demand.
std::mutex g_ws_mu;
std::unordered_map<int, std::pair<void *, size_t>> g_ws;

int cached_workspace(size_t need, void **ws) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return GDN_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_ws_mu);
    auto &slot = g_ws[dev];
    if (slot.second < need) {
        if (slot.first) {
            if (hipDeviceSynchronize() != hipSuccess) return GDN_ERR_HIP;
            if (hipFree(slot.first) != hipSuccess) return GDN_ERR_HIP;
            slot = {nullptr, 0};
        }
        void *ptr = nullptr;
        if (hipMalloc(&ptr, need) != hipSuccess) return GDN_ERR_HIP;
        slot = {ptr, need};
    }
    *ws = slot.first;
    return GDN_OK;
}

int run_cached(const void *q, const void *k, const void *v, const float *alpha, const float *beta,
               const float *state_in, void *out, float *state_out, int B, int H, int T, int Dk,
               int Dv, int chunk, bool bf16, void *stream) {
    const size_t esz = bf16 ? 2 : 4;
    int st = validate(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, esz);
    if (st != GDN_OK) return st;
    const size_t need =
        ws_layout(B, H, T, Dk, Dv, esz, resolve_group(num_chunks(T), (long long)B * H, Dv, 0, bf16)).total;
    void *ws = nullptr;
    st = cached_workspace(need, &ws);
    if (st != GDN_OK) return st;
    return run(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, bf16, 0, ws,
               need, stream, nullptr);
}

// Allocation-free path (gdn_chunk_forward_noalloc): the workspace is a
// file-scope device array, one copy per GPU.  In host code `scratch` names a
// host-side stand-in, not a device address; the address of each GPU's copy
// comes from hipGetSymbolAddress and is kept per device.
static __device__ __align__(256) unsigned char scratch[GDN_NOALLOC_MAX_WORKSPACE];

std::mutex g_scratch_mu;
std::unordered_map<int, void *> g_scratch;  // device -> its copy of `scratch`

int scratch_address(void **ptr) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return GDN_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    auto it = g_scratch.find(dev);
    if (it == g_scratch.end()) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return GDN_ERR_HIP;
        it = g_scratch.emplace(dev, p).first;
    }
    *ptr = it->second;
    return GDN_OK;
}

int run_noalloc(const void *q, const void *k, const void *v, const float *alpha, const float *beta,
                const float *state_in, void *out, float *state_out, int B, int H, int T, int Dk, int Dv,
                int chunk, void *stream) {
    int st = validate(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, 2);
    if (st != GDN_OK) return st;
    const size_t need =
        ws_layout(B, H, T, Dk, Dv, 2, resolve_group(num_chunks(T), (long long)B * H, Dv, 0, true)).total;
    if (need > GDN_NOALLOC_MAX_WORKSPACE) return GDN_ERR_WORKSPACE;
    void *ws = nullptr;
    st = scratch_address(&ws);
    if (st != GDN_OK) return st;
    return run(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, true, 0, ws,
               GDN_NOALLOC_MAX_WORKSPACE, stream, nullptr);
}

// ---------------------------------------------------------------------------
// Frame-wise path (gdn_frame_forward*): frame summaries, their reduction over
// token splits, the scan over frames, and the output; optionally with the
// normalizer state (gdn_frame_forward_norm*) and in the bidirectional form
// (gdn_frame_forward_bidir*).

struct FrameArgs {
    const void *q, *k, *v;
    const float *alpha, *beta, *state_in, *z_in;
    void *out;
    float *state_out, *z_out;
    int B, H, F, N, Dk, Dv;
    float key_scale, eps;
    bool bf16, norm, bidir;
    // the fused operator (gdn_frame_forward_fused*): q and k are the raw
    // projections; the remaining fields are its prologue and epilogue inputs
    bool fused;
    const void *gate, *w_o;
    const float *gain_q, *gain_k, *rope_freq;
    const int *rope_axis;
    float rms_eps;
    int lat_w, t0;
};

struct FrameWs {
    size_t PG, PA, Gf, Af, Hf, Hb, PGz, Gzf, FQT, FQH, FKT, FKH, Y, total;
};

int frame_blocks(int N) { return (N + 63) / 64; }

// Token splits per frame: a split is a whole number of 64-token blocks, and
// the library's choice (token_splits <= 0) is the largest count that keeps the
// summary workgroups (one per split) within one per CU (256), at least 1.
int frame_splits(long long units, int N, int token_splits) {
    const int nb = frame_blocks(N);
    int ns = token_splits;
    if (ns <= 0) ns = (int)(256 / units);
    if (ns > nb) ns = nb;
    if (ns < 1) ns = 1;
    const int per = (nb + ns - 1) / ns;   // blocks per split
    return (nb + per - 1) / per;          // no empty split
}

// One layout for every variant: the A tiles, the state fragments and the
// backward histories have room for the normalizer's extra 16-column tile; the
// histories are used by the bidirectional form only, the unrotated-key Gram
// fragments and their partials by the fused operator only.  The fused
// operator in fp32 also keeps its feature maps and gated readout (ntok_feat =
// its B F N H token rows; 0 otherwise).
FrameWs frame_ws_layout(int B, int H, int F, int Dk, int Dv, size_t esz, int NS, size_t ntok_feat = 0) {
    const size_t bhf = (size_t)B * H * F;
    const size_t DVn = (size_t)Dv + 16;
    FrameWs L;
    size_t off = 0;
    // partial sums only with several token splits
    const size_t np = NS > 1 ? (size_t)NS : 0;
    L.PG = off; off = align256(off + bhf * np * Dk * Dk * 4);
    L.PA = off; off = align256(off + bhf * np * Dk * DVn * 4);
    L.Gf = off; off = align256(off + bhf * Dk * Dk * esz);
    L.Af = off; off = align256(off + bhf * Dk * DVn * 4);
    L.Hf = off; off = align256(off + bhf * Dk * DVn * esz);
    L.Hb = off; off = align256(off + bhf * Dk * DVn * 4);
    L.PGz = off; off = align256(off + bhf * np * Dk * Dk * 4);
    L.Gzf = off; off = align256(off + bhf * Dk * Dk * esz);
    L.FQT = off; off = align256(off + ntok_feat * Dk * 4);
    L.FQH = off; off = align256(off + ntok_feat * Dk * 4);
    L.FKT = off; off = align256(off + ntok_feat * Dk * 4);
    L.FKH = off; off = align256(off + ntok_feat * Dk * 4);
    L.Y = off;   off = align256(off + ntok_feat * Dv * 4);
    L.total = off;
    return L;
}

// Token rows whose features the fp32 fused operator keeps in the workspace.
size_t frame_feat_rows(bool fused, bool bf16, int B, int H, int F, int N) {
    return (fused && !bf16) ? (size_t)B * H * F * N : 0;
}

// Output workgroups per (frame, head): about `wgs` workgroups in all, each a
// run of whole 16-token tiles, none empty.
void frame_out_split(long long units, int N, int wgs, int &OB, int &tpw) {
    const int ntf = (N + 15) / 16;
    long long ob = (wgs + units - 1) / units;
    if (ob > ntf) ob = ntf;
    tpw = (int)((ntf + ob - 1) / ob);
    OB = (ntf + tpw - 1) / tpw;
}

bool frame_shape_ok(int B, int H, int F, int N) {
    if (B < 1 || H < 1 || F < 1 || N < 1) return false;
    const long long bh = (long long)B * H;
    if (bh > 65535) return false;
    // token indices (and a split's end, up to 64 * F past the last token) fit in int
    if ((long long)F * N + 64LL * F + N > 0x7fffffffLL) return false;
    // grid sizes of the summary and output kernels stay below 2^31
    const long long units = bh * F;
    if (4LL * frame_blocks(N) * units > 0x7fffffffLL) return false;
    if (8LL * ((N + 15) / 16) * ((units + 7) / 8) > 0x7fffffffLL) return false;
    return true;
}

bool frame_dims_ok(int Dk, int Dv) { return (Dk == 64 || Dk == 128) && (Dv == 64 || Dv == 128); }

int frame_validate(const FrameArgs &a) {
    if (!a.q || !a.k || !a.v || !a.alpha || !a.beta || !a.out) return GDN_ERR_NULL;
    if (!frame_shape_ok(a.B, a.H, a.F, a.N)) return GDN_ERR_SHAPE;
    if (!frame_dims_ok(a.Dk, a.Dv)) return GDN_ERR_UNSUPPORTED;
    if (misaligned(a.q) || misaligned(a.k) || misaligned(a.v) || misaligned(a.alpha) || misaligned(a.beta) ||
        misaligned(a.state_in) || misaligned(a.out) || misaligned(a.state_out) ||
        (a.norm && (misaligned(a.z_in) || misaligned(a.z_out))))
        return GDN_ERR_ALIGN;
    const size_t esz = a.bf16 ? 2 : 4;
    const size_t ntok = (size_t)a.B * a.F * a.N * a.H;
    const Range rq = range(a.q, ntok * a.Dk * esz), rk = range(a.k, ntok * a.Dk * esz),
                rv = range(a.v, ntok * a.Dv * esz), ra = range(a.alpha, (size_t)a.B * a.F * a.H * 4),
                rb = range(a.beta, ntok * 4), ro = range(a.out, ntok * a.Dv * esz);
    const size_t sbytes = (size_t)a.B * a.H * a.Dk * a.Dv * 4, zbytes = (size_t)a.B * a.H * a.Dk * 4;
    const Range rsi = range(a.state_in, sbytes), rso = range(a.state_out, sbytes);
    const Range rzi = range(a.norm ? a.z_in : nullptr, zbytes), rzo = range(a.norm ? a.z_out : nullptr, zbytes);
    // outputs may not overlap the inputs or each other; a state may be updated
    // in place (the same buffer in and out)
    const Range ins[] = {rq, rk, rv, ra, rb, rsi, rzi};
    for (const Range &r : ins)
        if (ro.overlaps(r)) return GDN_ERR_ALIAS;
    // state_out may share state_in's buffer exactly (in-place update), z_out z_in's
    const Range *outs[] = {&rso, &rzo};
    for (int o = 0; o < 2; ++o) {
        const Range &r = *outs[o];
        if (!r.valid()) continue;
        const int own = o == 0 ? 5 : 6;
        for (int i = 0; i < 7; ++i) {
            if (!r.overlaps(ins[i])) continue;
            if (i != own || r.lo != ins[i].lo) return GDN_ERR_ALIAS;
        }
        if (r.overlaps(ro)) return GDN_ERR_ALIAS;
    }
    if (rso.overlaps(rzo)) return GDN_ERR_ALIAS;
    if (a.fused) {
        if (!a.gate || !a.w_o || !a.gain_q || !a.gain_k || !a.rope_freq || !a.rope_axis) return GDN_ERR_NULL;
        if (a.lat_w < 1) return GDN_ERR_SHAPE;
        if (!a.norm) return GDN_ERR_UNSUPPORTED;
        if (misaligned(a.gate) || misaligned(a.w_o) || misaligned(a.gain_q) || misaligned(a.gain_k) ||
            misaligned(a.rope_freq) || misaligned(a.rope_axis))
            return GDN_ERR_ALIGN;
        const Range extra[] = {range(a.gate, ntok * a.Dv * esz), range(a.w_o, (size_t)a.H * a.Dv * a.Dv * esz),
                               range(a.gain_q, (size_t)a.H * a.Dk * 4), range(a.gain_k, (size_t)a.H * a.Dk * 4),
                               range(a.rope_freq, (size_t)a.Dk / 2 * 4), range(a.rope_axis, (size_t)a.Dk / 2 * 4)};
        for (const Range &r : extra)
            if (ro.overlaps(r) || rso.overlaps(r) || rzo.overlaps(r)) return GDN_ERR_ALIAS;
    }
    return GDN_OK;
}

template <class E>
gdn::FrameParams<E> make_frame_params(const FrameArgs &a, int NS, void *ws) {
    gdn::FrameParams<E> p;
    p.q = (const E *)a.q;
    p.k = (const E *)a.k;
    p.v = (const E *)a.v;
    p.alpha = a.alpha;
    p.beta = a.beta;
    p.state_in = a.state_in;
    p.out = (E *)a.out;
    p.state_out = a.state_out;
    p.B = a.B;
    p.H = a.H;
    p.F = a.F;
    p.N = a.N;
    p.NS = NS;
    p.NBT = 64 * ((frame_blocks(a.N) + NS - 1) / NS);
    frame_out_split((long long)a.B * a.H * a.F, a.N, gdn::kFrameOutWgs, p.OB, p.OTPW);
    p.key_scale = a.key_scale;
    p.z_in = a.norm ? a.z_in : nullptr;
    p.z_out = a.norm ? a.z_out : nullptr;
    p.eps = a.eps;
    const FrameWs L = frame_ws_layout(a.B, a.H, a.F, a.Dk, a.Dv, sizeof(E), NS,
                                      frame_feat_rows(a.fused, a.bf16, a.B, a.H, a.F, a.N));
    unsigned char *base = (unsigned char *)ws;
    p.PG = (float *)(base + L.PG);
    p.PA = (float *)(base + L.PA);
    p.Gf = (E *)(base + L.Gf);
    p.Af = (float *)(base + L.Af);
    p.Hf = (E *)(base + L.Hf);
    p.Hb = (float *)(base + L.Hb);
    p.PGz = (float *)(base + L.PGz);
    p.Gzf = (E *)(base + L.Gzf);
    p.fqt = (float *)(base + L.FQT);
    p.fqh = (float *)(base + L.FQH);
    p.fkt = (float *)(base + L.FKT);
    p.fkh = (float *)(base + L.FKH);
    p.ybuf = (float *)(base + L.Y);
    p.sum_mode = 0;
    p.gate = (const E *)a.gate;
    p.w_o = (const E *)a.w_o;
    p.gain_q = a.gain_q;
    p.gain_k = a.gain_k;
    p.rope_freq = a.rope_freq;
    p.rope_axis = a.rope_axis;
    p.rms_eps = a.rms_eps;
    p.lat_w = a.lat_w;
    p.t0 = a.t0;
    p.feat_scale = a.key_scale;
    if (a.fused) {
        // the key scale is applied to the key features as they are formed
        p.key_scale = 1.f;
        // one workgroup per CU (the fused output needs 100+ KB of LDS): at
        // most 256 workgroups in all unless the units alone exceed that
        const long long units = (long long)a.B * a.H * a.F;
        const int ntf = (a.N + 15) / 16;
        long long ob = 256 / units;
        if (ob < 1) ob = 1;
        if (ob > ntf) ob = ntf;
        p.OTPW = (int)((ntf + ob - 1) / ob);
        p.OB = (ntf + p.OTPW - 1) / p.OTPW;
    }
    return p;
}

constexpr int kFrameStages = 4;  // summaries, reduction, scan, output

template <class E, int DK, int DV, bool NORM, bool BIDIR, bool FUSED = false>
hipError_t launch_frame(const gdn::FrameParams<E> &p, hipStream_t s, int reps, hipEvent_t *ev) {
    using LS = gdn::FrameSumLds<E, DK, DV, FUSED>;
    using LO = gdn::FrameOutLds<E, DK, DV, NORM>;
    using LF = gdn::FusedOutLds<DK, DV>;
    const void *out_kernel;
    size_t out_lds;
    if constexpr (FUSED) {
        out_kernel = (const void *)gdn::gdn_frame_output_fused_kernel<DK, DV>;
        out_lds = LF::bytes;
    } else {
        out_kernel = (const void *)gdn::gdn_frame_output_kernel<E, DK, DV, NORM>;
        out_lds = LO::bytes;
    }
    static std::once_flag attr_once;
    static hipError_t attr_err = hipSuccess;
    std::call_once(attr_once, [&] {
        hipError_t e = hipFuncSetAttribute((const void *)gdn::gdn_frame_summary_kernel<E, DK, DV, NORM, FUSED>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)LS::bytes);
        if (e == hipSuccess)
            e = hipFuncSetAttribute(out_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)out_lds);
        attr_err = e;
    });
    if (attr_err != hipSuccess) return attr_err;
    const long long BH = (long long)p.B * p.H, units = BH * p.F;
    constexpr int NJ = DV / 16 + NORM;
    // reduction items per unit (FUSED: also the unrotated-key G fragments)
    constexpr int NI = (DK / 16) * (DK / 32) * (FUSED ? 2 : 1) + (DK / 16) * NJ;
    auto stage = [&](int i) -> hipError_t {
        switch (i) {
        case 0:
            return launch((const void *)gdn::gdn_frame_summary_kernel<E, DK, DV, NORM, FUSED>,
                          dim3((unsigned)(units * p.NS)), dim3(gdn::sum_threads<FUSED>()), LS::bytes, s, p);
        case 1:
            // a single split writes the summaries in their final form
            if (p.NS > 1)
                return launch((const void *)gdn::gdn_frame_reduce_kernel<E, DK, DV, NORM, FUSED>,
                              dim3((unsigned)units, (NI + 3) / 4), dim3(256), 0, s, p);
            return hipSuccess;
        case 2:
            return launch((const void *)gdn::gdn_frame_scan_kernel<E, DK, DV, NORM, BIDIR, FUSED>,
                          dim3(gdn::xcd_blocks(BH, NJ)), dim3(64), 0, s, p);
        default:
            if constexpr (FUSED)
                return launch((const void *)gdn::gdn_frame_output_fused_kernel<DK, DV>,
                              dim3(gdn::xcd_blocks(units, p.OB)), dim3(gdn::kFusedOutWaves * 64), LF::bytes, s, p);
            else
                return launch((const void *)gdn::gdn_frame_output_kernel<E, DK, DV, NORM>,
                              dim3(gdn::xcd_blocks(units, p.OB)), dim3(LO::WAVES * 64), LO::bytes, s, p);
        }
    };
    hipError_t er = hipSuccess;
    for (int i = 0; i < kFrameStages && er == hipSuccess; ++i) {
        if (!ev) {
            er = stage(i);
            continue;
        }
        er = hipEventRecord(ev[2 * i], s);
        for (int r = 0; r < reps && er == hipSuccess; ++r) er = stage(i);
        if (er == hipSuccess) er = hipEventRecord(ev[2 * i + 1], s);
    }
    return er;
}

// The fused operator in fp32: features, then the summaries on the rotated keys
// (G, A) and on the unrotated ones (the normalizer's Gram matrix and K~^T beta),
// the fused reduction and scan, and the fp32 output and projection.  The four
// profiled stages are: features and summaries, reduction, scan, output and
// projection.
template <int DK, int DV, bool BIDIR>
hipError_t launch_frame_fused32(const gdn::FrameParams<float> &p, hipStream_t s, int reps, hipEvent_t *ev) {
    using E = float;
    using LS = gdn::FrameSumLds<E, DK, DV, false>;
    using LO = gdn::FrameOutLds<E, DK, DV, true>;
    using LP = gdn::ProjectLds<DV>;
    static std::once_flag attr_once;
    static hipError_t attr_err = hipSuccess;
    std::call_once(attr_once, [&] {
        hipError_t e = hipFuncSetAttribute((const void *)gdn::gdn_frame_summary_kernel<E, DK, DV, true, false>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)LS::bytes);
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)gdn::gdn_frame_output_f32_fused_kernel<DK, DV>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)LO::bytes);
        if (e == hipSuccess)
            e = hipFuncSetAttribute((const void *)gdn::gdn_frame_project_f32_kernel<DV>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)LP::bytes);
        attr_err = e;
    });
    if (attr_err != hipSuccess) return attr_err;
    const long long BH = (long long)p.B * p.H, units = BH * p.F;
    constexpr int NJ = DV / 16 + 1;
    constexpr int NI = (DK / 16) * (DK / 32) * 2 + (DK / 16) * NJ;
    const size_t rows = 2 * (size_t)BH * p.F * p.N;                 // q and k rows
    const size_t feat_blocks = (rows + 4 * (128 / DK) - 1) / (4 * (128 / DK));
    auto stage = [&](int i) -> hipError_t {
        switch (i) {
        case 0: {
            hipError_t e = launch((const void *)gdn::gdn_frame_features_kernel<DK>, dim3((unsigned)feat_blocks),
                                  dim3(256), 0, s, p);
            // rotated keys: G and the A tiles
            gdn::FrameParams<E> pr = p;
            pr.k = p.fkh;
            pr.sum_mode = 1;
            if (e == hipSuccess)
                e = launch((const void *)gdn::gdn_frame_summary_kernel<E, DK, DV, true, false>,
                           dim3((unsigned)(units * p.NS)), dim3(gdn::sum_threads<false>()), LS::bytes, s, pr);
            // unrotated keys: their Gram matrix into the unrotated-key regions, the normalizer tile
            gdn::FrameParams<E> pu = p;
            pu.k = p.fkt;
            pu.sum_mode = 2;
            pu.PG = p.PGz;
            pu.Gf = p.Gzf;
            if (e == hipSuccess)
                e = launch((const void *)gdn::gdn_frame_summary_kernel<E, DK, DV, true, false>,
                           dim3((unsigned)(units * p.NS)), dim3(gdn::sum_threads<false>()), LS::bytes, s, pu);
            return e;
        }
        case 1:
            if (p.NS > 1)
                return launch((const void *)gdn::gdn_frame_reduce_kernel<E, DK, DV, true, true>,
                              dim3((unsigned)units, (NI + 3) / 4), dim3(256), 0, s, p);
            return hipSuccess;
        case 2:
            return launch((const void *)gdn::gdn_frame_scan_kernel<E, DK, DV, true, BIDIR, true>,
                          dim3(gdn::xcd_blocks(BH, NJ)), dim3(64), 0, s, p);
        default: {
            hipError_t e = launch((const void *)gdn::gdn_frame_output_f32_fused_kernel<DK, DV>,
                                  dim3(gdn::xcd_blocks(units, p.OB)), dim3(LO::WAVES * 64), LO::bytes, s, p);
            if (e == hipSuccess)
                e = launch((const void *)gdn::gdn_frame_project_f32_kernel<DV>,
                           dim3((unsigned)(((size_t)p.F * p.N + 63) / 64), (unsigned)BH), dim3(256), LP::bytes, s, p);
            return e;
        }
        }
    };
    hipError_t er = hipSuccess;
    for (int i = 0; i < kFrameStages && er == hipSuccess; ++i) {
        if (!ev) {
            er = stage(i);
            continue;
        }
        er = hipEventRecord(ev[2 * i], s);
        for (int r = 0; r < reps && er == hipSuccess; ++r) er = stage(i);
        if (er == hipSuccess) er = hipEventRecord(ev[2 * i + 1], s);
    }
    return er;
}

template <bool BIDIR>
hipError_t frame_dispatch_fused32(const gdn::FrameParams<float> &p, int Dk, int Dv, hipStream_t s, int reps,
                                  hipEvent_t *ev) {
    if (Dk == 128 && Dv == 128) return launch_frame_fused32<128, 128, BIDIR>(p, s, reps, ev);
    if (Dk == 64 && Dv == 64) return launch_frame_fused32<64, 64, BIDIR>(p, s, reps, ev);
    if (Dk == 128 && Dv == 64) return launch_frame_fused32<128, 64, BIDIR>(p, s, reps, ev);
    return launch_frame_fused32<64, 128, BIDIR>(p, s, reps, ev);
}

template <class E, bool NORM, bool BIDIR, bool FUSED = false>
hipError_t frame_dispatch_n(const gdn::FrameParams<E> &p, int Dk, int Dv, hipStream_t s, int reps, hipEvent_t *ev) {
    if (Dk == 128 && Dv == 128) return launch_frame<E, 128, 128, NORM, BIDIR, FUSED>(p, s, reps, ev);
    if (Dk == 64 && Dv == 64) return launch_frame<E, 64, 64, NORM, BIDIR, FUSED>(p, s, reps, ev);
    if (Dk == 128 && Dv == 64) return launch_frame<E, 128, 64, NORM, BIDIR, FUSED>(p, s, reps, ev);
    return launch_frame<E, 64, 128, NORM, BIDIR, FUSED>(p, s, reps, ev);
}

template <class E>
hipError_t frame_dispatch(const FrameArgs &a, int NS, void *ws, hipStream_t s, int reps, hipEvent_t *ev) {
    const gdn::FrameParams<E> p = make_frame_params<E>(a, NS, ws);
    if constexpr (sizeof(E) == 2) {
        if (a.fused)
            return a.bidir ? frame_dispatch_n<E, true, true, true>(p, a.Dk, a.Dv, s, reps, ev)
                           : frame_dispatch_n<E, true, false, true>(p, a.Dk, a.Dv, s, reps, ev);
    } else {
        if (a.fused)
            return a.bidir ? frame_dispatch_fused32<true>(p, a.Dk, a.Dv, s, reps, ev)
                           : frame_dispatch_fused32<false>(p, a.Dk, a.Dv, s, reps, ev);
    }
    if (a.bidir)
        return a.norm ? frame_dispatch_n<E, true, true>(p, a.Dk, a.Dv, s, reps, ev)
                      : frame_dispatch_n<E, false, true>(p, a.Dk, a.Dv, s, reps, ev);
    return a.norm ? frame_dispatch_n<E, true, false>(p, a.Dk, a.Dv, s, reps, ev)
                  : frame_dispatch_n<E, false, false>(p, a.Dk, a.Dv, s, reps, ev);
}

int frame_run(const FrameArgs &a, int token_splits, void *ws, size_t ws_bytes, void *stream, int reps,
              hipEvent_t *ev) {
    int st = frame_validate(a);
    if (st != GDN_OK) return st;
    const int NS = frame_splits((long long)a.B * a.H * a.F, a.N, token_splits);
    if (!ws || ((uintptr_t)ws & 255u) ||
        ws_bytes < frame_ws_layout(a.B, a.H, a.F, a.Dk, a.Dv, a.bf16 ? 2 : 4, NS,
                                   frame_feat_rows(a.fused, a.bf16, a.B, a.H, a.F, a.N))
                       .total)
        return GDN_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    const hipError_t e = a.bf16 ? frame_dispatch<uint16_t>(a, NS, ws, s, reps, ev)
                                : frame_dispatch<float>(a, NS, ws, s, reps, ev);
    return e == hipSuccess ? GDN_OK : GDN_ERR_HIP;
}

int frame_run_cached(const FrameArgs &a, void *stream) {
    int st = frame_validate(a);
    if (st != GDN_OK) return st;
    const size_t need = frame_ws_layout(a.B, a.H, a.F, a.Dk, a.Dv, a.bf16 ? 2 : 4,
                                        frame_splits((long long)a.B * a.H * a.F, a.N, 0),
                                        frame_feat_rows(a.fused, a.bf16, a.B, a.H, a.F, a.N))
                            .total;
    void *ws = nullptr;
    st = cached_workspace(need, &ws);
    if (st != GDN_OK) return st;
    return frame_run(a, 0, ws, need, stream, 1, nullptr);
}

int frame_profile(const FrameArgs &a, int token_splits, void *ws, size_t ws_bytes, int reps, float *stage_ms,
                  void *stream) {
    if (!stage_ms || reps < 1) return GDN_ERR_NULL;
    // stages are re-run in place, so no state may be updated in place
    if (a.state_in && a.state_in == a.state_out) return GDN_ERR_ALIAS;
    if (a.norm && a.z_in && a.z_in == a.z_out) return GDN_ERR_ALIAS;
    hipEvent_t ev[2 * kFrameStages] = {};
    int status = GDN_OK;
    for (auto &e : ev)
        if (status == GDN_OK && hipEventCreate(&e) != hipSuccess) {
            e = nullptr;
            status = GDN_ERR_HIP;
        }
    if (status == GDN_OK) status = frame_run(a, token_splits, ws, ws_bytes, stream, reps, ev);
    if (status == GDN_OK && hipStreamSynchronize((hipStream_t)stream) != hipSuccess) status = GDN_ERR_HIP;
    for (int i = 0; i < kFrameStages && status == GDN_OK; ++i) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, ev[2 * i], ev[2 * i + 1]) != hipSuccess) status = GDN_ERR_HIP;
        stage_ms[i] = ms / reps;
    }
    for (auto &e : ev)
        if (e) (void)hipEventDestroy(e);
    return status;
}

FrameArgs frame_args(const void *q, const void *k, const void *v, const float *alpha, const float *beta,
                     const float *state_in, const float *z_in, void *out, float *state_out, float *z_out, int B,
                     int H, int F, int N, int Dk, int Dv, float key_scale, float eps, bool bf16, bool norm,
                     bool bidir = false) {
    return FrameArgs{q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out,
                     B, H, F, N, Dk, Dv, key_scale, eps, bf16, norm, bidir};
}

FrameArgs fused_args(const void *q_raw, const void *k_raw, const void *v, const void *gate, const void *w_o,
                     const float *alpha, const float *beta, const float *gain_q, const float *gain_k,
                     const float *rope_freq, const int *rope_axis, const float *state_in, const float *z_in,
                     void *out, float *state_out, float *z_out, int B, int H, int F, int N, int Dk, int Dv,
                     int lat_w, int t0, float key_scale, float rms_eps, float eps, int bidirectional,
                     bool bf16 = true) {
    FrameArgs a = frame_args(q_raw, k_raw, v, alpha, beta, state_in, z_in, out, state_out, z_out, B, H, F, N, Dk,
                             Dv, key_scale, eps, bf16, true, bidirectional != 0);
    a.fused = true;
    a.gate = gate;
    a.w_o = w_o;
    a.gain_q = gain_q;
    a.gain_k = gain_k;
    a.rope_freq = rope_freq;
    a.rope_axis = rope_axis;
    a.rms_eps = rms_eps;
    a.lat_w = lat_w;
    a.t0 = t0;
    return a;
}

}  // namespace

extern "C" {

int gdn_chunk_forward(const void *q, const void *k, const void *v, const float *alpha,
                      const float *beta, const float *state_in, void *out, float *state_out, int B,
                      int H, int T, int Dk, int Dv, int chunk, void *stream) {
    return run_cached(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, true,
                      stream);
}

int gdn_chunk_forward_f32(const float *q, const float *k, const float *v, const float *alpha,
                          const float *beta, const float *state_in, float *out, float *state_out,
                          int B, int H, int T, int Dk, int Dv, int chunk, void *stream) {
    return run_cached(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, false,
                      stream);
}

int gdn_workspace_check(int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16, int scan_group) {
    if (!shape_ok(B, H, T)) return GDN_ERR_SHAPE;
    if (!dims_ok(Dk, Dv, chunk)) return GDN_ERR_UNSUPPORTED;
    const size_t esz = is_bf16 ? 2 : 4;
    const int G = resolve_group(num_chunks(T), (long long)B * H, Dv, scan_group, is_bf16 != 0);
    const WsLayout L = ws_layout(B, H, T, Dk, Dv, esz, G);
    const WsNeeds n = ws_needs(B, H, T, Dk, Dv, esz, G);
    const size_t start[] = {L.g, L.gf, L.W, L.Ut, L.Hs, L.Us, L.Nf, L.PsiT, L.lgam, L.HgT, L.total};
    const size_t need[] = {n.g, n.gf, n.W, n.Ut, n.Hs, n.Us, n.Nf, n.PsiT, n.lgam, n.HgT};
    for (int r = 0; r < 10; ++r) {
        if (start[r] % 256) return r + 1;                    // regions start 256-byte aligned
        if (need[r] > start[r + 1] - start[r]) return r + 1;  // region too small
    }
    return GDN_OK;
}

int gdn_chunk_forward_noalloc(const void *q, const void *k, const void *v, const float *alpha,
                              const float *beta, const float *state_in, void *out, float *state_out, int B,
                              int H, int T, int Dk, int Dv, int chunk, void *stream) {
    return run_noalloc(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, stream);
}

size_t gdn_workspace_bytes(int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16) {
    return gdn_workspace_bytes_ex(B, H, T, Dk, Dv, chunk, is_bf16, 0);
}

int gdn_scan_group_size(int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16, int scan_group) {
    if (!shape_ok(B, H, T) || !dims_ok(Dk, Dv, chunk)) return 0;
    return resolve_group(num_chunks(T), (long long)B * H, Dv, scan_group, is_bf16 != 0);
}

size_t gdn_workspace_bytes_ex(int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16,
                              int scan_group) {
    if (!shape_ok(B, H, T) || !dims_ok(Dk, Dv, chunk)) return 0;
    return ws_layout(B, H, T, Dk, Dv, is_bf16 ? 2 : 4,
                     resolve_group(num_chunks(T), (long long)B * H, Dv, scan_group, is_bf16 != 0))
        .total;
}

int gdn_chunk_forward_ws(const void *q, const void *k, const void *v, const float *alpha,
                         const float *beta, const float *state_in, void *out, float *state_out,
                         int B, int H, int T, int Dk, int Dv, int chunk, void *ws, size_t ws_bytes,
                         void *stream) {
    return run(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, true, 0, ws,
               ws_bytes, stream, nullptr);
}

int gdn_chunk_forward_f32_ws(const float *q, const float *k, const float *v, const float *alpha,
                             const float *beta, const float *state_in, float *out, float *state_out,
                             int B, int H, int T, int Dk, int Dv, int chunk, void *ws,
                             size_t ws_bytes, void *stream) {
    return run(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, false, 0, ws,
               ws_bytes, stream, nullptr);
}

int gdn_chunk_forward_ex(const void *q, const void *k, const void *v, const float *alpha,
                         const float *beta, const float *state_in, void *out, float *state_out,
                         int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16, int scan_group,
                         void *ws, size_t ws_bytes, void *stream) {
    return run(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk, is_bf16 != 0,
               scan_group, ws, ws_bytes, stream, nullptr);
}

int gdn_profile_stages(const void *q, const void *k, const void *v, const float *alpha,
                       const float *beta, const float *state_in, void *out, float *state_out,
                       int B, int H, int T, int Dk, int Dv, int chunk, int is_bf16, int scan_group,
                       void *ws, size_t ws_bytes, int reps, float *stage_ms, void *stream) {
    if (!stage_ms || reps < 1) return GDN_ERR_NULL;
    // Stages are re-run in place, so the state may not be updated in place.
    if (state_in && state_in == state_out) return GDN_ERR_ALIAS;
    StageTiming tm{};
    tm.reps = reps;
    int status = GDN_OK;
    for (auto &e : tm.ev)
        if (status == GDN_OK && hipEventCreate(&e) != hipSuccess) {
            e = nullptr;
            status = GDN_ERR_HIP;
        }
    if (status == GDN_OK)
        status = run(q, k, v, alpha, beta, state_in, out, state_out, B, H, T, Dk, Dv, chunk,
                     is_bf16 != 0, scan_group, ws, ws_bytes, stream, &tm);
    if (status == GDN_OK && hipStreamSynchronize((hipStream_t)stream) != hipSuccess)
        status = GDN_ERR_HIP;
    for (int i = 0; i < kStages && status == GDN_OK; ++i) {
        float ms = 0.f;
        if (tm.ran[i] && hipEventElapsedTime(&ms, tm.ev[2 * i], tm.ev[2 * i + 1]) != hipSuccess)
            status = GDN_ERR_HIP;
        stage_ms[i] = tm.ran[i] ? ms / reps : 0.f;
    }
    for (auto &e : tm.ev)
        if (e) (void)hipEventDestroy(e);
    return status;
}

int gdn_frame_forward(const void *q, const void *k, const void *v, const float *alpha, const float *beta,
                      const float *state_in, void *out, float *state_out, int B, int H, int F, int N,
                      int Dk, int Dv, float key_scale, void *stream) {
    return frame_run_cached(frame_args(q, k, v, alpha, beta, state_in, nullptr, out, state_out, nullptr, B, H,
                                       F, N, Dk, Dv, key_scale, 0.f, true, false),
                            stream);
}

int gdn_frame_forward_f32(const float *q, const float *k, const float *v, const float *alpha,
                          const float *beta, const float *state_in, float *out, float *state_out, int B,
                          int H, int F, int N, int Dk, int Dv, float key_scale, void *stream) {
    return frame_run_cached(frame_args(q, k, v, alpha, beta, state_in, nullptr, out, state_out, nullptr, B, H,
                                       F, N, Dk, Dv, key_scale, 0.f, false, false),
                            stream);
}

int gdn_frame_token_splits(int B, int H, int F, int N, int Dk, int Dv, int token_splits) {
    if (!frame_shape_ok(B, H, F, N) || !frame_dims_ok(Dk, Dv)) return 0;
    return frame_splits((long long)B * H * F, N, token_splits);
}

size_t gdn_frame_workspace_bytes(int B, int H, int F, int N, int Dk, int Dv, int is_bf16, int token_splits) {
    if (!frame_shape_ok(B, H, F, N) || !frame_dims_ok(Dk, Dv)) return 0;
    return frame_ws_layout(B, H, F, Dk, Dv, is_bf16 ? 2 : 4, frame_splits((long long)B * H * F, N, token_splits))
        .total;
}

int gdn_frame_forward_ex(const void *q, const void *k, const void *v, const float *alpha, const float *beta,
                         const float *state_in, void *out, float *state_out, int B, int H, int F, int N,
                         int Dk, int Dv, float key_scale, int is_bf16, int token_splits, void *ws,
                         size_t ws_bytes, void *stream) {
    return frame_run(frame_args(q, k, v, alpha, beta, state_in, nullptr, out, state_out, nullptr, B, H, F, N,
                                Dk, Dv, key_scale, 0.f, is_bf16 != 0, false),
                     token_splits, ws, ws_bytes, stream, 1, nullptr);
}

int gdn_frame_profile_stages(const void *q, const void *k, const void *v, const float *alpha,
                             const float *beta, const float *state_in, void *out, float *state_out, int B,
                             int H, int F, int N, int Dk, int Dv, float key_scale, int is_bf16,
                             int token_splits, void *ws, size_t ws_bytes, int reps, float *stage_ms,
                             void *stream) {
    return frame_profile(frame_args(q, k, v, alpha, beta, state_in, nullptr, out, state_out, nullptr, B, H, F,
                                    N, Dk, Dv, key_scale, 0.f, is_bf16 != 0, false),
                         token_splits, ws, ws_bytes, reps, stage_ms, stream);
}

int gdn_frame_forward_norm(const void *q, const void *k, const void *v, const float *alpha, const float *beta,
                           const float *state_in, const float *z_in, void *out, float *state_out, float *z_out,
                           int B, int H, int F, int N, int Dk, int Dv, float key_scale, float eps, int is_bf16,
                           void *stream) {
    return frame_run_cached(frame_args(q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out, B, H, F, N,
                                       Dk, Dv, key_scale, eps, is_bf16 != 0, true),
                            stream);
}

int gdn_frame_forward_norm_ex(const void *q, const void *k, const void *v, const float *alpha,
                              const float *beta, const float *state_in, const float *z_in, void *out,
                              float *state_out, float *z_out, int B, int H, int F, int N, int Dk, int Dv,
                              float key_scale, float eps, int is_bf16, int token_splits, void *ws,
                              size_t ws_bytes, void *stream) {
    return frame_run(frame_args(q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out, B, H, F, N, Dk, Dv,
                                key_scale, eps, is_bf16 != 0, true),
                     token_splits, ws, ws_bytes, stream, 1, nullptr);
}

int gdn_frame_profile_stages_norm(const void *q, const void *k, const void *v, const float *alpha,
                                  const float *beta, const float *state_in, const float *z_in, void *out,
                                  float *state_out, float *z_out, int B, int H, int F, int N, int Dk, int Dv,
                                  float key_scale, float eps, int is_bf16, int token_splits, void *ws,
                                  size_t ws_bytes, int reps, float *stage_ms, void *stream) {
    return frame_profile(frame_args(q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out, B, H, F, N, Dk,
                                    Dv, key_scale, eps, is_bf16 != 0, true),
                         token_splits, ws, ws_bytes, reps, stage_ms, stream);
}

int gdn_frame_forward_bidir(const void *q, const void *k, const void *v, const float *alpha, const float *beta,
                            const float *state_in, const float *z_in, void *out, float *state_out,
                            float *z_out, int B, int H, int F, int N, int Dk, int Dv, float key_scale, float eps,
                            int is_bf16, int normalized, void *stream) {
    return frame_run_cached(frame_args(q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out, B, H, F, N,
                                       Dk, Dv, key_scale, eps, is_bf16 != 0, normalized != 0, true),
                            stream);
}

int gdn_frame_forward_bidir_ex(const void *q, const void *k, const void *v, const float *alpha,
                               const float *beta, const float *state_in, const float *z_in, void *out,
                               float *state_out, float *z_out, int B, int H, int F, int N, int Dk, int Dv,
                               float key_scale, float eps, int is_bf16, int normalized, int token_splits,
                               void *ws, size_t ws_bytes, void *stream) {
    return frame_run(frame_args(q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out, B, H, F, N, Dk, Dv,
                                key_scale, eps, is_bf16 != 0, normalized != 0, true),
                     token_splits, ws, ws_bytes, stream, 1, nullptr);
}

int gdn_frame_profile_stages_bidir(const void *q, const void *k, const void *v, const float *alpha,
                                   const float *beta, const float *state_in, const float *z_in, void *out,
                                   float *state_out, float *z_out, int B, int H, int F, int N, int Dk, int Dv,
                                   float key_scale, float eps, int is_bf16, int normalized, int token_splits,
                                   void *ws, size_t ws_bytes, int reps, float *stage_ms, void *stream) {
    return frame_profile(frame_args(q, k, v, alpha, beta, state_in, z_in, out, state_out, z_out, B, H, F, N, Dk,
                                    Dv, key_scale, eps, is_bf16 != 0, normalized != 0, true),
                         token_splits, ws, ws_bytes, reps, stage_ms, stream);
}

int gdn_frame_forward_fused(const void *q_raw, const void *k_raw, const void *v, const void *gate,
                            const void *w_o, const float *alpha, const float *beta, const float *gain_q,
                            const float *gain_k, const float *rope_freq, const int *rope_axis,
                            const float *state_in, const float *z_in, void *out, float *state_out, float *z_out,
                            int B, int H, int F, int N, int Dk, int Dv, int lat_w, int t0, float key_scale,
                            float rms_eps, float eps, int bidirectional, void *stream) {
    return frame_run_cached(fused_args(q_raw, k_raw, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq,
                                       rope_axis, state_in, z_in, out, state_out, z_out, B, H, F, N, Dk, Dv, lat_w,
                                       t0, key_scale, rms_eps, eps, bidirectional),
                            stream);
}

int gdn_frame_forward_fused_ex(const void *q_raw, const void *k_raw, const void *v, const void *gate,
                               const void *w_o, const float *alpha, const float *beta, const float *gain_q,
                               const float *gain_k, const float *rope_freq, const int *rope_axis,
                               const float *state_in, const float *z_in, void *out, float *state_out,
                               float *z_out, int B, int H, int F, int N, int Dk, int Dv, int lat_w, int t0,
                               float key_scale, float rms_eps, float eps, int bidirectional, int token_splits,
                               void *ws, size_t ws_bytes, void *stream) {
    return frame_run(fused_args(q_raw, k_raw, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq, rope_axis,
                                state_in, z_in, out, state_out, z_out, B, H, F, N, Dk, Dv, lat_w, t0, key_scale,
                                rms_eps, eps, bidirectional),
                     token_splits, ws, ws_bytes, stream, 1, nullptr);
}

int gdn_frame_profile_stages_fused(const void *q_raw, const void *k_raw, const void *v, const void *gate,
                                   const void *w_o, const float *alpha, const float *beta, const float *gain_q,
                                   const float *gain_k, const float *rope_freq, const int *rope_axis,
                                   const float *state_in, const float *z_in, void *out, float *state_out,
                                   float *z_out, int B, int H, int F, int N, int Dk, int Dv, int lat_w, int t0,
                                   float key_scale, float rms_eps, float eps, int bidirectional,
                                   int token_splits, void *ws, size_t ws_bytes, int reps, float *stage_ms,
                                   void *stream) {
    return frame_profile(fused_args(q_raw, k_raw, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq,
                                    rope_axis, state_in, z_in, out, state_out, z_out, B, H, F, N, Dk, Dv, lat_w, t0,
                                    key_scale, rms_eps, eps, bidirectional),
                         token_splits, ws, ws_bytes, reps, stage_ms, stream);
}

int gdn_frame_forward_fused_f32(const float *q_raw, const float *k_raw, const float *v, const float *gate,
                                const float *w_o, const float *alpha, const float *beta, const float *gain_q,
                                const float *gain_k, const float *rope_freq, const int *rope_axis,
                                const float *state_in, const float *z_in, float *out, float *state_out,
                                float *z_out, int B, int H, int F, int N, int Dk, int Dv, int lat_w, int t0,
                                float key_scale, float rms_eps, float eps, int bidirectional, void *stream) {
    return frame_run_cached(fused_args(q_raw, k_raw, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq,
                                       rope_axis, state_in, z_in, out, state_out, z_out, B, H, F, N, Dk, Dv, lat_w,
                                       t0, key_scale, rms_eps, eps, bidirectional, false),
                            stream);
}

int gdn_frame_forward_fused_f32_ex(const float *q_raw, const float *k_raw, const float *v, const float *gate,
                                   const float *w_o, const float *alpha, const float *beta, const float *gain_q,
                                   const float *gain_k, const float *rope_freq, const int *rope_axis,
                                   const float *state_in, const float *z_in, float *out, float *state_out,
                                   float *z_out, int B, int H, int F, int N, int Dk, int Dv, int lat_w, int t0,
                                   float key_scale, float rms_eps, float eps, int bidirectional, int token_splits,
                                   void *ws, size_t ws_bytes, void *stream) {
    return frame_run(fused_args(q_raw, k_raw, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq, rope_axis,
                                state_in, z_in, out, state_out, z_out, B, H, F, N, Dk, Dv, lat_w, t0, key_scale,
                                rms_eps, eps, bidirectional, false),
                     token_splits, ws, ws_bytes, stream, 1, nullptr);
}

int gdn_frame_profile_stages_fused_f32(const float *q_raw, const float *k_raw, const float *v, const float *gate,
                                       const float *w_o, const float *alpha, const float *beta,
                                       const float *gain_q, const float *gain_k, const float *rope_freq,
                                       const int *rope_axis, const float *state_in, const float *z_in, float *out,
                                       float *state_out, float *z_out, int B, int H, int F, int N, int Dk, int Dv,
                                       int lat_w, int t0, float key_scale, float rms_eps, float eps,
                                       int bidirectional, int token_splits, void *ws, size_t ws_bytes, int reps,
                                       float *stage_ms, void *stream) {
    return frame_profile(fused_args(q_raw, k_raw, v, gate, w_o, alpha, beta, gain_q, gain_k, rope_freq,
                                    rope_axis, state_in, z_in, out, state_out, z_out, B, H, F, N, Dk, Dv, lat_w, t0,
                                    key_scale, rms_eps, eps, bidirectional, false),
                         token_splits, ws, ws_bytes, reps, stage_ms, stream);
}

size_t gdn_frame_fused_workspace_bytes(int B, int H, int F, int N, int Dk, int Dv, int is_bf16, int token_splits) {
    if (!frame_shape_ok(B, H, F, N) || !frame_dims_ok(Dk, Dv)) return 0;
    return frame_ws_layout(B, H, F, Dk, Dv, is_bf16 ? 2 : 4, frame_splits((long long)B * H * F, N, token_splits),
                           frame_feat_rows(true, is_bf16 != 0, B, H, F, N))
        .total;
}

const char *gdn_status_string(int status) {
    switch (status) {
    case GDN_OK: return "ok";
    case GDN_ERR_NULL: return "a required pointer is NULL";
    case GDN_ERR_SHAPE: return "invalid shape (sizes must be >= 1, B*H <= 65535, token and grid indices within int range)";
    case GDN_ERR_UNSUPPORTED: return "unsupported configuration (Dk, Dv in {64,128}; chunk == 64)";
    case GDN_ERR_WORKSPACE: return "workspace missing, too small or not 256-byte aligned";
    case GDN_ERR_HIP: return "HIP runtime error or kernel launch failure";
    case GDN_ERR_ALIGN: return "a pointer is not 16-byte aligned";
    case GDN_ERR_ALIAS: return "an output overlaps an input";
    default: return "unknown status";
    }
}

}  // extern "C"
