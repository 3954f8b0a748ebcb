/*
 * Plain fp64 CPU oracle for the gated delta-rule (GDN) forward.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the correctness reference that the
 * GPU path is checked against.  It shares no code, header, table or helper
 * with the HIP library, and only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load it.  The product path never
 * calls it.
 *
 * What it computes (Section "Frame-wise Gated DeltaNet", subsection
 * "Frame-wise delta-rule update", equations appendix_gdn_kv_update and
 * appendix_gdn_kv_compact, taken with one token per update; the same update
 * is equation gdn_combined in Section "Hybrid Architecture"):
 *
 *   for every (b, h) independently, for t = 0 .. T-1:
 *       S~   = alpha_t * S_{t-1}                       (decay first)
 *       S_t  = S~ + beta_t (v_t - S~ k_t) k_t^T        (write only the residual)
 *       o_t  = S_t q_t                                 (read after the update)
 *
 * which equals S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T.
 * The paper's state S is Dv x Dk.  Here it is stored transposed,
 * H = S^T with shape [Dk][Dv] (row-major), the same orientation the paper's
 * kernel section uses when it left-multiplies the state.  In that orientation
 * the step reads:
 *       p   = H^T k            (prediction of v from the decayed state / alpha)
 *       H  <- alpha H + k (beta (v - alpha p))^T
 *       o   = H^T q
 * Only the terminal state is returned, as the streaming cache carries it
 * (subsection "Streaming cache").
 *
 * Everything is computed in double precision.  Inputs are read in their
 * stored type and widened exactly (bf16 -> fp64 is a 16-bit shift), so no
 * rounded copy of the inputs is ever made.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_F64 = 2 };

static double load_elem(const void *p, int dtype, size_t i)
{
    if (dtype == ORC_F32)
        return (double)((const float *)p)[i];
    if (dtype == ORC_BF16) {
        uint32_t u = (uint32_t)((const uint16_t *)p)[i] << 16;
        float f;
        memcpy(&f, &u, sizeof f);
        return (double)f;
    }
    return ((const double *)p)[i];
}

struct job {
    const void *q, *k, *v;
    int qkv_dtype;
    const void *alpha, *beta, *state_in;
    int gate_dtype, state_dtype;
    double *out, *state_out;
    int B, H, T, Dk, Dv;
    int nthreads;
    int worker;
    int status;
};

static int run_head(const struct job *J, int b, int h)
{
    const int H = J->H, T = J->T, Dk = J->Dk, Dv = J->Dv;
    double *S = (double *)calloc((size_t)Dk * Dv, sizeof(double));
    double *kk = (double *)malloc(sizeof(double) * (size_t)Dk);
    double *qq = (double *)malloc(sizeof(double) * (size_t)Dk);
    double *vv = (double *)malloc(sizeof(double) * (size_t)Dv);
    double *p = (double *)malloc(sizeof(double) * (size_t)Dv);
    if (!S || !kk || !qq || !vv || !p) {
        free(S); free(kk); free(qq); free(vv); free(p);
        return -1;
    }
    const size_t sbase = ((size_t)b * H + h) * (size_t)Dk * Dv;
    if (J->state_in) {
        for (size_t e = 0; e < (size_t)Dk * Dv; e++)
            S[e] = load_elem(J->state_in, J->state_dtype, sbase + e);
    }
    for (int t = 0; t < T; t++) {
        const size_t row = ((size_t)b * T + t) * H + h;
        for (int i = 0; i < Dk; i++) {
            kk[i] = load_elem(J->k, J->qkv_dtype, row * Dk + i);
            qq[i] = load_elem(J->q, J->qkv_dtype, row * Dk + i);
        }
        for (int j = 0; j < Dv; j++)
            vv[j] = load_elem(J->v, J->qkv_dtype, row * Dv + j);
        const double a = load_elem(J->alpha, J->gate_dtype, row);
        const double be = load_elem(J->beta, J->gate_dtype, row);

        /* p = H^T k : what the undecayed state predicts for v */
        for (int j = 0; j < Dv; j++)
            p[j] = 0.0;
        for (int i = 0; i < Dk; i++)
            for (int j = 0; j < Dv; j++)
                p[j] += S[(size_t)i * Dv + j] * kk[i];
        /* residual of the decayed state, scaled by the write gate */
        for (int j = 0; j < Dv; j++)
            p[j] = be * (vv[j] - a * p[j]);
        /* H <- alpha H + k r^T */
        for (int i = 0; i < Dk; i++)
            for (int j = 0; j < Dv; j++)
                S[(size_t)i * Dv + j] = a * S[(size_t)i * Dv + j] + kk[i] * p[j];
        /* o_t = S_t q_t = H^T q, read from the updated state */
        double *o = J->out + row * Dv;
        for (int j = 0; j < Dv; j++)
            o[j] = 0.0;
        for (int i = 0; i < Dk; i++)
            for (int j = 0; j < Dv; j++)
                o[j] += S[(size_t)i * Dv + j] * qq[i];
    }
    if (J->state_out)
        memcpy(J->state_out + sbase, S, sizeof(double) * (size_t)Dk * Dv);
    free(S); free(kk); free(qq); free(vv); free(p);
    return 0;
}

static void *worker_main(void *arg)
{
    struct job *J = (struct job *)arg;
    const int nbh = J->B * J->H;
    for (int bh = J->worker; bh < nbh; bh += J->nthreads) {
        if (run_head(J, bh / J->H, bh % J->H) != 0) {
            J->status = -1;
            break;
        }
    }
    return NULL;
}

/*
 * q, k : [B, T, H, Dk]   v : [B, T, H, Dv]     stored as qkv_dtype (0 f32, 1 bf16 bits, 2 f64)
 * alpha, beta : [B, T, H]                      stored as gate_dtype (0 f32, 2 f64)
 * state_in : [B, H, Dk, Dv] or NULL (zero)     stored as state_dtype (0 f32, 2 f64)
 * out : [B, T, H, Dv] fp64 (required)          state_out : [B, H, Dk, Dv] fp64 or NULL
 * nthreads : worker threads over the (b, h) streams (< 1 means 1)
 * Returns 0, or -1 on bad arguments / allocation failure.
 */
int gdn_oracle_forward(const void *q, const void *k, const void *v, int qkv_dtype,
                       const void *alpha, const void *beta, int gate_dtype,
                       const void *state_in, int state_dtype,
                       double *out, double *state_out,
                       int B, int H, int T, int Dk, int Dv, int nthreads)
{
    if (!q || !k || !v || !alpha || !beta || !out)
        return -1;
    if (B < 1 || H < 1 || T < 0 || Dk < 1 || Dv < 1)
        return -1;
    if (qkv_dtype < 0 || qkv_dtype > 2 || (gate_dtype != 0 && gate_dtype != 2) ||
        (state_dtype != 0 && state_dtype != 2))
        return -1;
    const int nbh = B * H;
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > nbh)
        nthreads = nbh;

    struct job *jobs = (struct job *)calloc((size_t)nthreads, sizeof(struct job));
    pthread_t *tids = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    char *running = (char *)calloc((size_t)nthreads, 1);
    if (!jobs || !tids || !running) {
        free(jobs); free(tids); free(running);
        return -1;
    }
    int status = 0;
    for (int w = 0; w < nthreads; w++) {
        struct job *J = &jobs[w];
        J->q = q; J->k = k; J->v = v; J->qkv_dtype = qkv_dtype;
        J->alpha = alpha; J->beta = beta; J->gate_dtype = gate_dtype;
        J->state_in = state_in; J->state_dtype = state_dtype;
        J->out = out; J->state_out = state_out;
        J->B = B; J->H = H; J->T = T; J->Dk = Dk; J->Dv = Dv;
        J->nthreads = nthreads; J->worker = w; J->status = 0;
        if (nthreads > 1 && pthread_create(&tids[w], NULL, worker_main, J) == 0)
            running[w] = 1;
        else
            worker_main(J); /* single thread, or a thread could not start */
    }
    for (int w = 0; w < nthreads; w++)
        if (running[w])
            pthread_join(tids[w], NULL);
    for (int w = 0; w < nthreads; w++)
        if (jobs[w].status)
            status = -1;
    free(running);
    free(jobs);
    free(tids);
    return status;
}

/*
 * Frame-wise form (the paper's own update: Section "Frame-wise Gated
 * DeltaNet", equations appendix_gdn_kv_update / appendix_gdn_kv_compact with a
 * frame of N tokens; eq. gdn_combined): one decay alpha_f per frame and head,
 * shared by the frame's N tokens, which all write at once; a write gate beta
 * per token; the keys rescaled by key_scale before entering the recurrence
 * (the paper uses 1/sqrt(D N), subsection "Attention features").  With the
 * keys k~ = key_scale k, in the H = S^T orientation, per frame f:
 *       p_n  = H^T k~_n                  for every token n of the frame (old H)
 *       u_n  = beta_n (v_n - alpha_f p_n)
 *       H   <- alpha_f H + sum_n k~_n u_n^T
 *       o_n  = H^T q_n                   (read from the updated state)
 * i.e. S_f = alpha_f S_{f-1} (I - K~ B K~^T) + V B K~^T and Y_f = S_f Q_f.
 *
 * With the normalizer (subsection "Frame-wise delta-rule update", equation
 * appendix_gdn_z_update; subsection "Normalized readout and output
 * projection", equation appendix_gdn_readout), a vector state z = S^z of
 * length Dk is carried beside H and updated in the same correction-based way
 * from the (unrotated) keys:
 *       z~   = alpha_f z                     (decay first)
 *       z   <- z~ + sum_n beta_n (1 - k~_n . z~) k~_n
 *       o_n  = (H^T q_n) / (z . q_n + eps)   (both from the updated states)
 * This path has no rotary embedding, so the rotated and unrotated keys and
 * queries coincide.
 *
 * Bidirectional (the paper's bidirectional GDN: a forward scan from the
 * cache plus a backward scan within the call started from zero, Algorithm
 * alg:gdn-kernel, Phase B; the two histories are added before the readout):
 * the backward state of frame f is the same frame recurrence run over the
 * later frames F-1, F-2, .., f+1 of the call from a zero state (and z = 0),
 *       Hb_{F-1} = 0,   Hb_{f-1} = frame f's update applied to Hb_f,
 * and every readout of frame f uses H_f + Hb_f (and z_f + zb_f).  Only the
 * forward terminal state is returned, as the cache carries it.
 */
struct fjob {
    const void *q, *k, *v;
    int qkv_dtype;
    const void *alpha, *beta, *state_in;
    int gate_dtype, state_dtype;
    double *out, *state_out;
    int B, H, F, N, Dk, Dv;
    double key_scale;
    int norm;                      /* 1: carry z and divide the readout */
    int bidir;                     /* 1: add the backward history to every readout */
    const void *z_in;              /* [B][H][Dk] or NULL, stored as state_dtype */
    double *z_out;                 /* [B][H][Dk] or NULL */
    double eps;
    int nthreads, worker, status;
};

/* One frame's update of (S, z) in place: decay, then the simultaneous
 * residual write of the frame's N tokens (kk, uu, zr are scratch). */
static void frame_update(const struct fjob *J, int b, int h, int f, double *S, double *z, double *kk,
                         double *uu, double *zr)
{
    const int H = J->H, F = J->F, N = J->N, Dk = J->Dk, Dv = J->Dv;
    const size_t T = (size_t)F * N;
    const double a = load_elem(J->alpha, J->gate_dtype, ((size_t)b * F + f) * H + h);
    for (int n = 0; n < N; n++) {
        const size_t row = ((size_t)b * T + (size_t)f * N + n) * H + h;
        const double be = load_elem(J->beta, J->gate_dtype, row);
        double *kn = kk + (size_t)n * Dk, *un = uu + (size_t)n * Dv;
        for (int i = 0; i < Dk; i++)
            kn[i] = J->key_scale * load_elem(J->k, J->qkv_dtype, row * Dk + i);
        for (int j = 0; j < Dv; j++)
            un[j] = 0.0;
        for (int i = 0; i < Dk; i++)
            for (int j = 0; j < Dv; j++)
                un[j] += S[(size_t)i * Dv + j] * kn[i];
        for (int j = 0; j < Dv; j++)
            un[j] = be * (load_elem(J->v, J->qkv_dtype, row * Dv + j) - a * un[j]);
        if (J->norm) {
            double dot = 0.0;
            for (int i = 0; i < Dk; i++)
                dot += kn[i] * z[i];
            zr[n] = be * (1.0 - a * dot);
        }
    }
    for (size_t e = 0; e < (size_t)Dk * Dv; e++)
        S[e] *= a;
    for (int n = 0; n < N; n++) {
        const double *kn = kk + (size_t)n * Dk, *un = uu + (size_t)n * Dv;
        for (int i = 0; i < Dk; i++)
            for (int j = 0; j < Dv; j++)
                S[(size_t)i * Dv + j] += kn[i] * un[j];
    }
    if (J->norm) {
        for (int i = 0; i < Dk; i++)
            z[i] *= a;
        for (int n = 0; n < N; n++)
            for (int i = 0; i < Dk; i++)
                z[i] += zr[n] * kk[(size_t)n * Dk + i];
    }
}

static int run_frame_head(const struct fjob *J, int b, int h)
{
    const int H = J->H, F = J->F, N = J->N, Dk = J->Dk, Dv = J->Dv;
    const size_t T = (size_t)F * N;
    const size_t SD = (size_t)Dk * Dv;
    double *S = (double *)calloc(SD, sizeof(double));
    double *kk = (double *)malloc(sizeof(double) * (size_t)N * Dk);
    double *uu = (double *)malloc(sizeof(double) * (size_t)N * Dv);
    double *qq = (double *)malloc(sizeof(double) * (size_t)Dk);
    double *z = (double *)calloc((size_t)Dk, sizeof(double));
    double *zr = (double *)malloc(sizeof(double) * (size_t)N);
    /* bidirectional: the backward histories of every frame */
    double *Sb = J->bidir ? (double *)calloc((size_t)F * SD, sizeof(double)) : NULL;
    double *zb = J->bidir ? (double *)calloc((size_t)F * Dk, sizeof(double)) : NULL;
    if (!S || !kk || !uu || !qq || !z || !zr || (J->bidir && (!Sb || !zb))) {
        free(S); free(kk); free(uu); free(qq); free(z); free(zr); free(Sb); free(zb);
        return -1;
    }
    const size_t sbase = ((size_t)b * H + h) * SD;
    const size_t zbase = ((size_t)b * H + h) * (size_t)Dk;
    if (J->bidir) {
        /* backward scan within the call, from zero: Sb[F-1] = 0 and
         * Sb[f-1] = frame f's update applied to Sb[f] */
        for (int f = F - 1; f >= 1; f--) {
            memcpy(Sb + (size_t)(f - 1) * SD, Sb + (size_t)f * SD, sizeof(double) * SD);
            memcpy(zb + (size_t)(f - 1) * Dk, zb + (size_t)f * Dk, sizeof(double) * (size_t)Dk);
            frame_update(J, b, h, f, Sb + (size_t)(f - 1) * SD, zb + (size_t)(f - 1) * Dk, kk, uu, zr);
        }
    }
    if (J->state_in)
        for (size_t e = 0; e < SD; e++)
            S[e] = load_elem(J->state_in, J->state_dtype, sbase + e);
    if (J->norm && J->z_in)
        for (int i = 0; i < Dk; i++)
            z[i] = load_elem(J->z_in, J->state_dtype, zbase + i);
    for (int f = 0; f < F; f++) {
        frame_update(J, b, h, f, S, z, kk, uu, zr);
        /* readout from the updated state (plus the backward history) */
        const double *Sf = J->bidir ? Sb + (size_t)f * SD : NULL;
        const double *zf = J->bidir ? zb + (size_t)f * Dk : NULL;
        for (int n = 0; n < N; n++) {
            const size_t row = ((size_t)b * T + (size_t)f * N + n) * H + h;
            for (int i = 0; i < Dk; i++)
                qq[i] = load_elem(J->q, J->qkv_dtype, row * Dk + i);
            double *o = J->out + row * Dv;
            for (int j = 0; j < Dv; j++)
                o[j] = 0.0;
            for (int i = 0; i < Dk; i++)
                for (int j = 0; j < Dv; j++)
                    o[j] += (Sf ? S[(size_t)i * Dv + j] + Sf[(size_t)i * Dv + j] : S[(size_t)i * Dv + j]) * qq[i];
            if (J->norm) {
                double d = 0.0;
                for (int i = 0; i < Dk; i++)
                    d += (zf ? z[i] + zf[i] : z[i]) * qq[i];
                for (int j = 0; j < Dv; j++)
                    o[j] /= d + J->eps;
            }
        }
    }
    if (J->state_out)
        memcpy(J->state_out + sbase, S, sizeof(double) * SD);
    if (J->norm && J->z_out)
        memcpy(J->z_out + zbase, z, sizeof(double) * (size_t)Dk);
    free(S); free(kk); free(uu); free(qq); free(z); free(zr); free(Sb); free(zb);
    return 0;
}

static void *frame_worker_main(void *arg)
{
    struct fjob *J = (struct fjob *)arg;
    const int nbh = J->B * J->H;
    for (int bh = J->worker; bh < nbh; bh += J->nthreads) {
        if (run_frame_head(J, bh / J->H, bh % J->H) != 0) {
            J->status = -1;
            break;
        }
    }
    return NULL;
}

/*
 * q, k : [B, F*N, H, Dk]   v : [B, F*N, H, Dv]   stored as qkv_dtype (0 f32, 1 bf16 bits, 2 f64)
 * alpha : [B, F, H] (one per frame)   beta : [B, F*N, H]   stored as gate_dtype (0 f32, 2 f64)
 * state_in : [B, H, Dk, Dv] or NULL (zero)   out : [B, F*N, H, Dv] fp64   state_out : fp64 or NULL
 * key_scale : factor applied to every key (the paper's 1/sqrt(D N))
 * Returns 0, or -1 on bad arguments / allocation failure.
 */
static int frame_forward_impl(const void *q, const void *k, const void *v, int qkv_dtype,
                              const void *alpha, const void *beta, int gate_dtype,
                              const void *state_in, const void *z_in, int state_dtype,
                              double *out, double *state_out, double *z_out,
                              int B, int H, int F, int N, int Dk, int Dv, double key_scale,
                              int norm, double eps, int bidir, int nthreads)
{
    if (!q || !k || !v || !alpha || !beta || !out)
        return -1;
    if (B < 1 || H < 1 || F < 0 || N < 1 || Dk < 1 || Dv < 1)
        return -1;
    if (qkv_dtype < 0 || qkv_dtype > 2 || (gate_dtype != 0 && gate_dtype != 2) ||
        (state_dtype != 0 && state_dtype != 2))
        return -1;
    const int nbh = B * H;
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > nbh)
        nthreads = nbh;
    struct fjob *jobs = (struct fjob *)calloc((size_t)nthreads, sizeof(struct fjob));
    pthread_t *tids = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    char *running = (char *)calloc((size_t)nthreads, 1);
    if (!jobs || !tids || !running) {
        free(jobs); free(tids); free(running);
        return -1;
    }
    int status = 0;
    for (int w = 0; w < nthreads; w++) {
        struct fjob *J = &jobs[w];
        J->q = q; J->k = k; J->v = v; J->qkv_dtype = qkv_dtype;
        J->alpha = alpha; J->beta = beta; J->gate_dtype = gate_dtype;
        J->state_in = state_in; J->state_dtype = state_dtype;
        J->out = out; J->state_out = state_out;
        J->B = B; J->H = H; J->F = F; J->N = N; J->Dk = Dk; J->Dv = Dv;
        J->key_scale = key_scale;
        J->norm = norm; J->z_in = z_in; J->z_out = z_out; J->eps = eps; J->bidir = bidir;
        J->nthreads = nthreads; J->worker = w; J->status = 0;
        if (nthreads > 1 && pthread_create(&tids[w], NULL, frame_worker_main, J) == 0)
            running[w] = 1;
        else
            frame_worker_main(J);
    }
    for (int w = 0; w < nthreads; w++)
        if (running[w])
            pthread_join(tids[w], NULL);
    for (int w = 0; w < nthreads; w++)
        if (jobs[w].status)
            status = -1;
    free(running);
    free(jobs);
    free(tids);
    return status;
}

int gdn_oracle_frame_forward(const void *q, const void *k, const void *v, int qkv_dtype,
                             const void *alpha, const void *beta, int gate_dtype,
                             const void *state_in, int state_dtype,
                             double *out, double *state_out,
                             int B, int H, int F, int N, int Dk, int Dv, double key_scale, int nthreads)
{
    return frame_forward_impl(q, k, v, qkv_dtype, alpha, beta, gate_dtype, state_in, NULL, state_dtype,
                              out, state_out, NULL, B, H, F, N, Dk, Dv, key_scale, 0, 0.0, 0, nthreads);
}

/*
 * The frame-wise forward with the normalizer state and the normalized readout
 * (see the comment above struct fjob).  Arguments as gdn_oracle_frame_forward,
 * plus z_in : [B, H, Dk] stored as state_dtype or NULL (zero), z_out : [B, H, Dk]
 * fp64 or NULL, and eps (the paper uses 1e-6).
 */
int gdn_oracle_frame_forward_norm(const void *q, const void *k, const void *v, int qkv_dtype,
                                  const void *alpha, const void *beta, int gate_dtype,
                                  const void *state_in, const void *z_in, int state_dtype,
                                  double *out, double *state_out, double *z_out,
                                  int B, int H, int F, int N, int Dk, int Dv, double key_scale,
                                  double eps, int nthreads)
{
    return frame_forward_impl(q, k, v, qkv_dtype, alpha, beta, gate_dtype, state_in, z_in, state_dtype,
                              out, state_out, z_out, B, H, F, N, Dk, Dv, key_scale, 1, eps, 0, nthreads);
}

/*
 * General form: normalized (0/1, z_in/z_out/eps used only with 1) and
 * bidirectional (0/1: every readout adds the backward history of the call,
 * see the comment above struct fjob).
 */
int gdn_oracle_frame_forward_ex(const void *q, const void *k, const void *v, int qkv_dtype,
                                const void *alpha, const void *beta, int gate_dtype,
                                const void *state_in, const void *z_in, int state_dtype,
                                double *out, double *state_out, double *z_out,
                                int B, int H, int F, int N, int Dk, int Dv, double key_scale,
                                int normalized, double eps, int bidirectional, int nthreads)
{
    return frame_forward_impl(q, k, v, qkv_dtype, alpha, beta, gate_dtype, state_in, z_in, state_dtype,
                              out, state_out, z_out, B, H, F, N, Dk, Dv, key_scale, normalized != 0, eps,
                              bidirectional != 0, nthreads);
}


/*
 * The whole GDN operator of one block around the frame recurrence, with its
 * prologue and epilogue (appendix on the GDN block: subsection "Attention
 * features" for the feature maps and the key rescale, subsection "Frame-wise
 * delta-rule update" for the two states, subsection "Normalized readout and
 * output projection", equations appendix_gdn_readout and
 * appendix_gdn_output; Algorithm alg:gdn-kernel lists the same steps).  Per
 * token n and head h, from the raw projections q_n, k_n (length Dk):
 *
 *   RMSNorm   r(x)  = gain (x) x / sqrt(mean_i x_i^2 + rms_eps)   (per token, over Dk)
 *   features  q~ = ReLU(r_q(q_n)),   k~ = key_scale ReLU(r_k(k_n))    (unrotated)
 *   3D RoPE   q^ = R_n q~,           k^ = R_n k~                     (rotated)
 *
 * R_n rotates every channel pair (2i, 2i+1) by the angle
 * theta_i = freq_i * c_{axis_i}(n), the coordinate of token n along the pair's
 * axis: token n = f N + s of the call has t = t0 + f (axis 0),
 * y = s / lat_w (axis 1) and x = s % lat_w (axis 2), and
 *       (x_2i, x_2i+1) -> (x_2i cos - x_2i+1 sin,  x_2i sin + x_2i+1 cos).
 *
 * The KV state takes the rotated keys and the normalizer the unrotated ones,
 * each in the correction-based frame update (decay, then the residual write):
 *       H <- alpha H + sum_n k^_n (beta_n (v_n - alpha H^T k^_n))^T
 *       z <- alpha z + sum_n k~_n  beta_n (1 - alpha k~_n . z)
 * the readout divides the rotated numerator by the unrotated denominator,
 *       y_n = (H^T q^_n) / (z . q~_n + eps),
 * and the epilogue gates it channel by channel and projects it per head:
 *       out_n = W_o (SiLU(gate_n) o y_n),   SiLU(x) = x / (1 + e^-x),
 * with out_n[i] = sum_j W_o[h][i][j] (SiLU(gate_n[j]) y_n[j]).  Bidirectional:
 * as above (the backward histories, from zero over the later frames, are added
 * to both states before the readout).
 */
struct ujob {
    const void *q, *k, *v, *gate, *w_o;
    int qkv_dtype;
    const void *alpha, *beta, *state_in, *z_in;
    int gate_dtype, state_dtype;
    const double *gain_q, *gain_k, *freq;     /* [H][Dk], [H][Dk], [Dk/2] */
    const int *axis;                          /* [Dk/2] in {0, 1, 2} */
    double rms_eps, key_scale, eps;
    int lat_w, t0, bidir;
    double *out, *state_out, *z_out;
    int B, H, F, N, Dk, Dv;
    int nthreads, worker, status;
};

/* Unrotated features of one token (RMSNorm with the head's gain, ReLU, times
 * scale) into xt and their rotation into xh. */
static void fused_features(const struct ujob *J, const void *src, size_t row, int h, const double *gain,
                           double scale, int f, int s, double *xt, double *xh)
{
    const int Dk = J->Dk;
    double ms = 0.0;
    for (int i = 0; i < Dk; i++) {
        const double x = load_elem(src, J->qkv_dtype, row * Dk + i);
        ms += x * x;
    }
    const double inv = 1.0 / sqrt(ms / Dk + J->rms_eps);
    for (int i = 0; i < Dk; i++) {
        const double x = gain[(size_t)h * Dk + i] * load_elem(src, J->qkv_dtype, row * Dk + i) * inv;
        xt[i] = scale * (x > 0.0 ? x : 0.0);
    }
    const double coord[3] = {(double)(J->t0 + f), (double)(s / J->lat_w), (double)(s % J->lat_w)};
    for (int i = 0; i < Dk / 2; i++) {
        const double th = J->freq[i] * coord[J->axis[i]];
        const double c = cos(th), sn = sin(th);
        xh[2 * i] = xt[2 * i] * c - xt[2 * i + 1] * sn;
        xh[2 * i + 1] = xt[2 * i] * sn + xt[2 * i + 1] * c;
    }
}

/* One frame's update of (S, z): the keys' features are formed here (kt
 * unrotated, kh rotated; uu, zr scratch). */
static void fused_update(const struct ujob *J, int b, int h, int f, double *S, double *z, double *kt, double *kh,
                         double *uu, double *zr)
{
    const int H = J->H, F = J->F, N = J->N, Dk = J->Dk, Dv = J->Dv;
    const size_t T = (size_t)F * N;
    const double a = load_elem(J->alpha, J->gate_dtype, ((size_t)b * F + f) * H + h);
    for (int n = 0; n < N; n++) {
        const size_t row = ((size_t)b * T + (size_t)f * N + n) * H + h;
        const double be = load_elem(J->beta, J->gate_dtype, row);
        double *ktn = kt + (size_t)n * Dk, *khn = kh + (size_t)n * Dk, *un = uu + (size_t)n * Dv;
        fused_features(J, J->k, row, h, J->gain_k, J->key_scale, f, n, ktn, khn);
        for (int j = 0; j < Dv; j++)
            un[j] = 0.0;
        for (int i = 0; i < Dk; i++)
            for (int j = 0; j < Dv; j++)
                un[j] += S[(size_t)i * Dv + j] * khn[i];
        for (int j = 0; j < Dv; j++)
            un[j] = be * (load_elem(J->v, J->qkv_dtype, row * Dv + j) - a * un[j]);
        double dot = 0.0;
        for (int i = 0; i < Dk; i++)
            dot += ktn[i] * z[i];
        zr[n] = be * (1.0 - a * dot);
    }
    for (size_t e = 0; e < (size_t)Dk * Dv; e++)
        S[e] *= a;
    for (int i = 0; i < Dk; i++)
        z[i] *= a;
    for (int n = 0; n < N; n++) {
        const double *khn = kh + (size_t)n * Dk, *ktn = kt + (size_t)n * Dk, *un = uu + (size_t)n * Dv;
        for (int i = 0; i < Dk; i++)
            for (int j = 0; j < Dv; j++)
                S[(size_t)i * Dv + j] += khn[i] * un[j];
        for (int i = 0; i < Dk; i++)
            z[i] += zr[n] * ktn[i];
    }
}

static int run_fused_head(const struct ujob *J, int b, int h)
{
    const int H = J->H, F = J->F, N = J->N, Dk = J->Dk, Dv = J->Dv;
    const size_t T = (size_t)F * N, SD = (size_t)Dk * Dv;
    double *S = (double *)calloc(SD, sizeof(double));
    double *z = (double *)calloc((size_t)Dk, sizeof(double));
    double *kt = (double *)malloc(sizeof(double) * (size_t)N * Dk);
    double *kh = (double *)malloc(sizeof(double) * (size_t)N * Dk);
    double *uu = (double *)malloc(sizeof(double) * (size_t)N * Dv);
    double *zr = (double *)malloc(sizeof(double) * (size_t)N);
    double *qt = (double *)malloc(sizeof(double) * (size_t)Dk);
    double *qh = (double *)malloc(sizeof(double) * (size_t)Dk);
    double *y = (double *)malloc(sizeof(double) * (size_t)Dv);
    double *Sb = J->bidir ? (double *)calloc((size_t)F * SD, sizeof(double)) : NULL;
    double *zb = J->bidir ? (double *)calloc((size_t)F * Dk, sizeof(double)) : NULL;
    int rc = -1;
    if (!S || !z || !kt || !kh || !uu || !zr || !qt || !qh || !y || (J->bidir && (!Sb || !zb)))
        goto done;
    const size_t sbase = ((size_t)b * H + h) * SD, zbase = ((size_t)b * H + h) * (size_t)Dk;
    if (J->bidir)
        for (int f = F - 1; f >= 1; f--) {
            memcpy(Sb + (size_t)(f - 1) * SD, Sb + (size_t)f * SD, sizeof(double) * SD);
            memcpy(zb + (size_t)(f - 1) * Dk, zb + (size_t)f * Dk, sizeof(double) * (size_t)Dk);
            fused_update(J, b, h, f, Sb + (size_t)(f - 1) * SD, zb + (size_t)(f - 1) * Dk, kt, kh, uu, zr);
        }
    if (J->state_in)
        for (size_t e = 0; e < SD; e++)
            S[e] = load_elem(J->state_in, J->state_dtype, sbase + e);
    if (J->z_in)
        for (int i = 0; i < Dk; i++)
            z[i] = load_elem(J->z_in, J->state_dtype, zbase + i);
    for (int f = 0; f < F; f++) {
        fused_update(J, b, h, f, S, z, kt, kh, uu, zr);
        const double *Sf = J->bidir ? Sb + (size_t)f * SD : NULL;
        const double *zf = J->bidir ? zb + (size_t)f * Dk : NULL;
        for (int n = 0; n < N; n++) {
            const size_t row = ((size_t)b * T + (size_t)f * N + n) * H + h;
            fused_features(J, J->q, row, h, J->gain_q, 1.0, f, n, qt, qh);
            double d = 0.0;
            for (int i = 0; i < Dk; i++)
                d += (zf ? z[i] + zf[i] : z[i]) * qt[i];
            for (int j = 0; j < Dv; j++)
                y[j] = 0.0;
            for (int i = 0; i < Dk; i++)
                for (int j = 0; j < Dv; j++)
                    y[j] += (Sf ? S[(size_t)i * Dv + j] + Sf[(size_t)i * Dv + j] : S[(size_t)i * Dv + j]) * qh[i];
            for (int j = 0; j < Dv; j++) {
                const double g = load_elem(J->gate, J->qkv_dtype, row * Dv + j);
                y[j] = g / (1.0 + exp(-g)) * (y[j] / (d + J->eps));
            }
            double *o = J->out + row * Dv;
            for (int i = 0; i < Dv; i++) {
                double acc = 0.0;
                for (int j = 0; j < Dv; j++)
                    acc += load_elem(J->w_o, J->qkv_dtype, ((size_t)h * Dv + i) * Dv + j) * y[j];
                o[i] = acc;
            }
        }
    }
    if (J->state_out)
        memcpy(J->state_out + sbase, S, sizeof(double) * SD);
    if (J->z_out)
        memcpy(J->z_out + zbase, z, sizeof(double) * (size_t)Dk);
    rc = 0;
done:
    free(S); free(z); free(kt); free(kh); free(uu); free(zr); free(qt); free(qh); free(y); free(Sb); free(zb);
    return rc;
}

static void *fused_worker_main(void *arg)
{
    struct ujob *J = (struct ujob *)arg;
    const int nbh = J->B * J->H;
    for (int bh = J->worker; bh < nbh; bh += J->nthreads)
        if (run_fused_head(J, bh / J->H, bh % J->H) != 0) {
            J->status = -1;
            break;
        }
    return NULL;
}

/*
 * q_raw, k_raw : [B, F*N, H, Dk]   v, gate : [B, F*N, H, Dv]   w_o : [H, Dv, Dv]
 *     (all stored as qkv_dtype: 0 f32, 1 bf16 bits, 2 f64)
 * alpha : [B, F, H]   beta : [B, F*N, H]   (gate_dtype 0 f32, 2 f64)
 * state_in [B, H, Dk, Dv], z_in [B, H, Dk] or NULL (zero), stored as state_dtype
 * gain_q, gain_k : [H, Dk] fp64   freq : [Dk/2] fp64   axis : [Dk/2] int in {0, 1, 2}
 * lat_w >= 1 (tokens per latent row), t0 (time coordinate of the first frame)
 * out : [B, F*N, H, Dv] fp64   state_out / z_out fp64 or NULL
 * Returns 0, or -1 on bad arguments / allocation failure.
 */
int gdn_oracle_frame_forward_fused(const void *q_raw, const void *k_raw, const void *v, const void *gate,
                                   const void *w_o, int qkv_dtype,
                                   const void *alpha, const void *beta, int gate_dtype,
                                   const void *state_in, const void *z_in, int state_dtype,
                                   const double *gain_q, const double *gain_k, double rms_eps,
                                   const double *freq, const int *axis, int lat_w, int t0,
                                   double *out, double *state_out, double *z_out,
                                   int B, int H, int F, int N, int Dk, int Dv, double key_scale, double eps,
                                   int bidirectional, int nthreads)
{
    if (!q_raw || !k_raw || !v || !gate || !w_o || !alpha || !beta || !gain_q || !gain_k || !freq || !axis ||
        !out)
        return -1;
    if (B < 1 || H < 1 || F < 0 || N < 1 || Dk < 2 || (Dk & 1) || Dv < 1 || lat_w < 1)
        return -1;
    if (qkv_dtype < 0 || qkv_dtype > 2 || (gate_dtype != 0 && gate_dtype != 2) ||
        (state_dtype != 0 && state_dtype != 2))
        return -1;
    for (int i = 0; i < Dk / 2; i++)
        if (axis[i] < 0 || axis[i] > 2)
            return -1;
    const int nbh = B * H;
    if (nthreads < 1)
        nthreads = 1;
    if (nthreads > nbh)
        nthreads = nbh;
    struct ujob *jobs = (struct ujob *)calloc((size_t)nthreads, sizeof(struct ujob));
    pthread_t *tids = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
    char *running = (char *)calloc((size_t)nthreads, 1);
    if (!jobs || !tids || !running) {
        free(jobs); free(tids); free(running);
        return -1;
    }
    for (int w = 0; w < nthreads; w++) {
        struct ujob *J = &jobs[w];
        J->q = q_raw; J->k = k_raw; J->v = v; J->gate = gate; J->w_o = w_o; J->qkv_dtype = qkv_dtype;
        J->alpha = alpha; J->beta = beta; J->gate_dtype = gate_dtype;
        J->state_in = state_in; J->z_in = z_in; J->state_dtype = state_dtype;
        J->gain_q = gain_q; J->gain_k = gain_k; J->freq = freq; J->axis = axis;
        J->rms_eps = rms_eps; J->key_scale = key_scale; J->eps = eps;
        J->lat_w = lat_w; J->t0 = t0; J->bidir = bidirectional != 0;
        J->out = out; J->state_out = state_out; J->z_out = z_out;
        J->B = B; J->H = H; J->F = F; J->N = N; J->Dk = Dk; J->Dv = Dv;
        J->nthreads = nthreads; J->worker = w; J->status = 0;
        if (nthreads > 1 && pthread_create(&tids[w], NULL, fused_worker_main, J) == 0)
            running[w] = 1;
        else
            fused_worker_main(J);
    }
    int status = 0;
    for (int w = 0; w < nthreads; w++)
        if (running[w])
            pthread_join(tids[w], NULL);
    for (int w = 0; w < nthreads; w++)
        if (jobs[w].status)
            status = -1;
    free(running);
    free(jobs);
    free(tids);
    return status;
}
