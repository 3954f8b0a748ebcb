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
