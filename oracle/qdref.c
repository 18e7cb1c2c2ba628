/*
 * Q-Delta CPU oracle: plain fp64 token-by-token recurrence and its exact
 * gradient by back-propagation through time.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the parity oracle for the GPU path.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load it.  It shares no code with the HIP kernels and must never be used as a
 * fallback for them.
 *
 * What it computes (paper: Sec. 3.3 "Q-Delta: Query-Aware Delta Rule",
 * Eq. (qdelta_decay), with the mixed input of Eq. (qdelta_gated_form)).
 * For every sequence n and head h independently, with state
 * S in R^{dv x dk} (row index = value component, column index = key component):
 *
 *     x_t = k_t + lambda_t q_t
 *     S_t = alpha_t S_{t-1} (I - beta_t x_t k_t^T) + beta_t v_t k_t^T
 *     o_t = S_t q_t                       (read-out uses the updated state)
 *
 * alpha == NULL means alpha_t = 1 for all t (the undecayed rule,
 * Eq. (qdelta_linear_form)).  The update is evaluated literally in the
 * expanded form  S_t = alpha_t S_{t-1} - alpha_t beta_t (S_{t-1} x_t) k_t^T
 *                      + beta_t v_t k_t^T,
 * i.e. S_{t-1} x_t is formed first (the "mixed prediction" of Sec. 3.2) and the
 * rank-one correction is applied to every entry.
 *
 * Gradients: exact gradients of
 *     L = sum_t <dO_t, o_t> + <dS_final, S_T>
 * with respect to q, k, v, beta, lambda, alpha and S_0, obtained by walking the
 * recurrence backwards (chain rule applied to the three lines above).  The
 * paper does not state a backward pass; this one is the plain derivative of
 * the recurrence.  Entry states are checkpointed every SEG tokens and each
 * segment is recomputed forward before it is walked backwards.
 *
 * Layouts (packed varlen form; a dense [B,T,...] batch is the special case
 * cu_seqlens = {0, T, 2T, ...}):
 *   q, k   [Ttot, H, dk]      v, o  [Ttot, H, dv]
 *   beta, lam, alpha          [Ttot, H]
 *   S0, S_final               [N, H, dv, dk]   (S0 == NULL means zero)
 * Work is split over (sequence, head) units on `nthreads` POSIX threads.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define SEG 64

typedef struct {
    int N, H, dk, dv;
    const int64_t *cu;
    const double *q, *k, *v, *beta, *lam, *alpha, *S0;
    /* forward outputs */
    double *o, *Sfin;
    /* backward inputs / outputs */
    const double *dO, *dSfin;
    double *dq, *dk_, *dv_, *dbeta, *dlam, *dalpha, *dS0;
    int do_bwd;
    int next;            /* next unit to take, guarded by mu */
    pthread_mutex_t mu;
} job_t;

static int take_unit(job_t *J) {
    pthread_mutex_lock(&J->mu);
    int u = J->next++;
    pthread_mutex_unlock(&J->mu);
    return u;
}

/* One recurrence step: S <- alpha S (I - beta x k^T) + beta v k^T.
 * Also returns p = S_{t-1} x (needed by the backward pass) in p[dv]. */
static void step(double *S, int dk, int dv, const double *qt, const double *kt,
                 const double *vt, double beta, double lam, double alpha,
                 double *x, double *p) {
    for (int j = 0; j < dk; ++j) x[j] = kt[j] + lam * qt[j];
    for (int i = 0; i < dv; ++i) {
        double s = 0.0;
        const double *Si = S + (size_t)i * dk;
        for (int j = 0; j < dk; ++j) s += Si[j] * x[j];
        p[i] = s;
    }
    for (int i = 0; i < dv; ++i) {
        double *Si = S + (size_t)i * dk;
        double e = beta * (vt[i] - alpha * p[i]);   /* beta (v - alpha S x) */
        for (int j = 0; j < dk; ++j) Si[j] = alpha * Si[j] + e * kt[j];
    }
}

static void readout(const double *S, int dk, int dv, const double *qt, double *ot) {
    for (int i = 0; i < dv; ++i) {
        double s = 0.0;
        const double *Si = S + (size_t)i * dk;
        for (int j = 0; j < dk; ++j) s += Si[j] * qt[j];
        ot[i] = s;
    }
}

static void run_unit(job_t *J, int unit) {
    const int H = J->H, dk = J->dk, dv = J->dv;
    const int n = unit / H, h = unit % H;
    const int64_t t0 = J->cu[n], t1 = J->cu[n + 1];
    const int64_t len = t1 - t0;
    const size_t SS = (size_t)dv * dk;

    double *S = (double *)calloc(SS, sizeof(double));
    double *x = (double *)malloc(sizeof(double) * dk);
    double *p = (double *)malloc(sizeof(double) * dv);
    if (J->S0) memcpy(S, J->S0 + ((size_t)n * H + h) * SS, SS * sizeof(double));

#define IDXK(t) ((((size_t)(t)) * H + h) * dk)
#define IDXV(t) ((((size_t)(t)) * H + h) * dv)
#define IDXG(t) (((size_t)(t)) * H + h)
#define ALPHA(t) (J->alpha ? J->alpha[IDXG(t)] : 1.0)

    if (!J->do_bwd) {
        for (int64_t t = t0; t < t1; ++t) {
            step(S, dk, dv, J->q + IDXK(t), J->k + IDXK(t), J->v + IDXV(t),
                 J->beta[IDXG(t)], J->lam[IDXG(t)], ALPHA(t), x, p);
            if (J->o) readout(S, dk, dv, J->q + IDXK(t), J->o + IDXV(t));
        }
        if (J->Sfin) memcpy(J->Sfin + ((size_t)n * H + h) * SS, S, SS * sizeof(double));
        free(S); free(x); free(p);
        return;
    }

    /* ---- backward: checkpoint entry states of every SEG-token segment ---- */
    const int64_t nseg = (len + SEG - 1) / SEG;
    double *ckpt = (double *)malloc(sizeof(double) * SS * (nseg > 0 ? nseg : 1));
    for (int64_t s = 0; s < nseg; ++s) {
        memcpy(ckpt + s * SS, S, SS * sizeof(double));
        int64_t a = t0 + s * SEG, b = a + SEG < t1 ? a + SEG : t1;
        for (int64_t t = a; t < b; ++t)
            step(S, dk, dv, J->q + IDXK(t), J->k + IDXK(t), J->v + IDXV(t),
                 J->beta[IDXG(t)], J->lam[IDXG(t)], ALPHA(t), x, p);
    }
    /* S is now S_T.  G accumulates dL/dS_t. */
    double *G = (double *)calloc(SS, sizeof(double));
    if (J->dSfin) memcpy(G, J->dSfin + ((size_t)n * H + h) * SS, SS * sizeof(double));

    /* per-segment stored states S_{t-1} for t in segment, plus p and x */
    double *Sprev = (double *)malloc(sizeof(double) * SS * SEG);
    double *Ps = (double *)malloc(sizeof(double) * dv * SEG);
    double *Xs = (double *)malloc(sizeof(double) * dk * SEG);
    double *Scur = (double *)malloc(sizeof(double) * SS);
    double *e = (double *)malloc(sizeof(double) * dv);
    double *de = (double *)malloc(sizeof(double) * dv);
    double *dp = (double *)malloc(sizeof(double) * dv);
    double *dx = (double *)malloc(sizeof(double) * dk);
    double *Gk = (double *)malloc(sizeof(double) * dv);

    for (int64_t s = nseg - 1; s >= 0; --s) {
        int64_t a = t0 + s * SEG, b = a + SEG < t1 ? a + SEG : t1;
        memcpy(Scur, ckpt + s * SS, SS * sizeof(double));
        for (int64_t t = a; t < b; ++t) {
            memcpy(Sprev + (t - a) * SS, Scur, SS * sizeof(double));
            step(Scur, dk, dv, J->q + IDXK(t), J->k + IDXK(t), J->v + IDXV(t),
                 J->beta[IDXG(t)], J->lam[IDXG(t)], ALPHA(t), Xs + (t - a) * dk,
                 Ps + (t - a) * dv);
        }
        /* Scur == S_{b-1} (state after the segment's last token) */
        for (int64_t t = b - 1; t >= a; --t) {
            const double *qt = J->q + IDXK(t), *kt = J->k + IDXK(t), *vt = J->v + IDXV(t);
            const double bt = J->beta[IDXG(t)], lt = J->lam[IDXG(t)], at = ALPHA(t);
            const double *Sp = Sprev + (t - a) * SS;   /* S_{t-1} */
            const double *pt = Ps + (t - a) * dv;       /* S_{t-1} x_t */
            const double *xt = Xs + (t - a) * dk;
            const double *dOt = J->dO ? J->dO + IDXV(t) : NULL;
            double *dqt = J->dq + IDXK(t), *dkt = J->dk_ + IDXK(t), *dvt = J->dv_ + IDXV(t);

            /* S_t for the read-out gradient: recompute from S_{t-1} */
            /* S_t = alpha S_{t-1} + (beta (v - alpha p)) k^T */
            for (int i = 0; i < dv; ++i) e[i] = vt[i] - at * pt[i];

            /* o_t = S_t q_t :  dS_t += dO_t q_t^T ;  dq_t = S_t^T dO_t */
            for (int j = 0; j < dk; ++j) dqt[j] = 0.0;
            if (dOt) {
                for (int i = 0; i < dv; ++i) {
                    const double *Spi = Sp + (size_t)i * dk;
                    double *Gi = G + (size_t)i * dk;
                    const double c = bt * e[i];
                    for (int j = 0; j < dk; ++j) {
                        double st = at * Spi[j] + c * kt[j];
                        dqt[j] += st * dOt[i];
                        Gi[j] += dOt[i] * qt[j];
                    }
                }
            }
            /* S_t = alpha S_{t-1} + beta e k^T  with  e = v - alpha p */
            /* Gk = G k */
            for (int i = 0; i < dv; ++i) {
                const double *Gi = G + (size_t)i * dk;
                double s = 0.0;
                for (int j = 0; j < dk; ++j) s += Gi[j] * kt[j];
                Gk[i] = s;
            }
            double dbt = 0.0;
            for (int i = 0; i < dv; ++i) dbt += e[i] * Gk[i];      /* e^T G k */
            for (int i = 0; i < dv; ++i) de[i] = bt * Gk[i];       /* beta G k */
            for (int j = 0; j < dk; ++j) dkt[j] = 0.0;
            for (int i = 0; i < dv; ++i) {                          /* beta G^T e */
                const double *Gi = G + (size_t)i * dk;
                const double c = bt * e[i];
                for (int j = 0; j < dk; ++j) dkt[j] += c * Gi[j];
            }
            double dat = 0.0;                                       /* <G, S_{t-1}> */
            for (size_t z = 0; z < SS; ++z) dat += G[z] * Sp[z];
            for (int i = 0; i < dv; ++i) {
                dvt[i] = de[i];                                     /* de/dv = I */
                dat -= pt[i] * de[i];                               /* e = v - alpha p */
                dp[i] = -at * de[i];
            }
            /* p = S_{t-1} x :  dx = S_{t-1}^T dp */
            for (int j = 0; j < dk; ++j) dx[j] = 0.0;
            for (int i = 0; i < dv; ++i) {
                const double *Spi = Sp + (size_t)i * dk;
                for (int j = 0; j < dk; ++j) dx[j] += Spi[j] * dp[i];
            }
            /* x = k + lambda q */
            double dlt = 0.0;
            for (int j = 0; j < dk; ++j) {
                dkt[j] += dx[j];
                dqt[j] += lt * dx[j];
                dlt += qt[j] * dx[j];
            }
            J->dbeta[IDXG(t)] = dbt;
            J->dlam[IDXG(t)] = dlt;
            if (J->dalpha) J->dalpha[IDXG(t)] = dat;
            /* dL/dS_{t-1} = alpha G + dp x^T */
            for (int i = 0; i < dv; ++i) {
                double *Gi = G + (size_t)i * dk;
                for (int j = 0; j < dk; ++j) Gi[j] = at * Gi[j] + dp[i] * xt[j];
            }
        }
    }
    if (J->dS0) memcpy(J->dS0 + ((size_t)n * H + h) * SS, G, SS * sizeof(double));
    if (J->Sfin) memcpy(J->Sfin + ((size_t)n * H + h) * SS, S, SS * sizeof(double));
    if (J->o) {
        /* forward outputs are also produced on request: rerun cheaply */
        memset(S, 0, SS * sizeof(double));
        if (J->S0) memcpy(S, J->S0 + ((size_t)n * H + h) * SS, SS * sizeof(double));
        for (int64_t t = t0; t < t1; ++t) {
            step(S, dk, dv, J->q + IDXK(t), J->k + IDXK(t), J->v + IDXV(t),
                 J->beta[IDXG(t)], J->lam[IDXG(t)], ALPHA(t), x, p);
            readout(S, dk, dv, J->q + IDXK(t), J->o + IDXV(t));
        }
    }
    free(ckpt); free(G); free(Sprev); free(Ps); free(Xs); free(Scur);
    free(e); free(de); free(dp); free(dx); free(Gk);
    free(S); free(x); free(p);
#undef IDXK
#undef IDXV
#undef IDXG
#undef ALPHA
}

static void *worker(void *arg) {
    job_t *J = (job_t *)arg;
    const int units = J->N * J->H;
    for (;;) {
        int u = take_unit(J);
        if (u >= units) break;
        run_unit(J, u);
    }
    return NULL;
}

static int run(job_t *J, int nthreads) {
    if (J->N < 0 || J->H <= 0 || J->dk <= 0 || J->dv <= 0 || !J->cu) return 1;
    for (int n = 0; n < J->N; ++n)
        if (J->cu[n + 1] < J->cu[n]) return 1;
    if (nthreads < 1) nthreads = 1;
    J->next = 0;
    pthread_mutex_init(&J->mu, NULL);
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * nthreads);
    int started = 0;
    for (int i = 0; i < nthreads; ++i)
        if (pthread_create(&th[i], NULL, worker, J) == 0) ++started;
    if (started == 0) worker(J);
    for (int i = 0; i < started; ++i) pthread_join(th[i], NULL);
    free(th);
    pthread_mutex_destroy(&J->mu);
    return 0;
}

/* Forward: o (may be NULL) and S_final (may be NULL).  Returns 0 on success. */
int qdref_fwd(int N, const int64_t *cu_seqlens, int H, int dk, int dv,
              const double *q, const double *k, const double *v,
              const double *beta, const double *lam, const double *alpha,
              const double *S0, double *o, double *S_final, int nthreads) {
    job_t J;
    memset(&J, 0, sizeof J);
    J.N = N; J.H = H; J.dk = dk; J.dv = dv; J.cu = cu_seqlens;
    J.q = q; J.k = k; J.v = v; J.beta = beta; J.lam = lam; J.alpha = alpha; J.S0 = S0;
    J.o = o; J.Sfin = S_final;
    return run(&J, nthreads);
}

/* Backward: gradients of <dO, o> + <dS_final, S_T>.  dO and dS_final may be
 * NULL (treated as zero).  dalpha and dS0 may be NULL (not computed).
 * dalpha is the gradient with respect to alpha itself (not log alpha). */
int qdref_bwd(int N, const int64_t *cu_seqlens, int H, int dk, int dv,
              const double *q, const double *k, const double *v,
              const double *beta, const double *lam, const double *alpha,
              const double *S0, const double *dO, const double *dS_final,
              double *dq, double *dk_, double *dv_, double *dbeta, double *dlam,
              double *dalpha, double *dS0, int nthreads) {
    job_t J;
    memset(&J, 0, sizeof J);
    J.N = N; J.H = H; J.dk = dk; J.dv = dv; J.cu = cu_seqlens;
    J.q = q; J.k = k; J.v = v; J.beta = beta; J.lam = lam; J.alpha = alpha; J.S0 = S0;
    J.dO = dO; J.dSfin = dS_final;
    J.dq = dq; J.dk_ = dk_; J.dv_ = dv_; J.dbeta = dbeta; J.dlam = dlam;
    J.dalpha = dalpha; J.dS0 = dS0;
    J.do_bwd = 1;
    return run(&J, nthreads);
}
