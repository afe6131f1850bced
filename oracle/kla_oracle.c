/*
 * kla_oracle.c -- fp64 sequential reference of the Kalman Linear Attention filter.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test-suite, the smoke check and the CPU baseline
 * leg of the benchmark do.  It shares no code with the GPU path.
 *
 * What it computes (paper: Sec. 4.2 "Parallel Inference via Moebius and Affine
 * Scans", Theorem 1 with its gate view, Theorem 2, and Appendix A's state-
 * expanded matrix form, eqs. kla-prec-mat / kla-mean-mat, with the readout
 * of Algorithm 1):
 *
 *   for every batch b, head h, key slot n and value channel d an independent
 *   scalar information filter runs over t = 1..T:
 *       rho    = 1 / (abar_t[n]^2 + pbar_t[n] * lam[n,d])        (prior ratio)
 *       lam    = rho * lam + k_t[n]^2 * Lv_t[d]                   (Theorem 1)
 *       eta    = abar_t[n] * rho * eta + k_t[n] * Lv_t[d] * v_t[d] (Theorem 2)
 *   and the readouts contract over the key slot (Algorithm 1):
 *       y_t[d]    = sum_n q_t[n] * eta[n,d] / lam[n,d]
 *       yvar_t[d] = sum_n q_t[n]^2 / lam[n,d]
 *
 * The value precision Lv is taken per (token, head, value channel), i.e. the
 * literal (B,T,1,D) shape of Algorithm 1; the precision lam is then an N x D
 * array per head, exactly as in eq. kla-prec-mat.  A caller that has one
 * scalar precision per (token, head) broadcasts it over d; every lam[n, :]
 * then coincides.
 *
 * No scan, chunking, exp/log factorisation or reassociation is used: this is
 * the recursion itself, token after token, in double precision.
 *
 * The backward pass is the exact reverse-mode derivative of that recursion
 * (the paper gives none).  Because the readout only couples filters through a
 * sum over n, the adjoint of each scalar filter's mean is known up front
 * (dL/dmu_t[n,d] = q_t[n] * dy_t[d]), so each (n, d) filter is differentiated
 * on its own: one forward sweep storing its (lam, eta) trajectory, then one
 * reverse sweep.  The readout variance is differentiable too (the Monte Carlo
 * readout of the paper's appendix samples through it): an upstream gradient
 * dyvar_t[d] adds 2 q dyvar / lam to dq and -q^2 dyvar / lam^2 to the adjoint
 * of lam_t.
 *
 * Layouts (all row-major, contiguous, double):
 *   q, k, a, p  [B, T, H, dk]       v, Lv, y, yvar, dy   [B, T, H, dv]
 *   lam0, eta0, lamT, etaT, dlamT, detaT, dlam0, deta0    [B, H, dk, dv]
 *
 * Gates per (n, d) (the *_nd entry points): Algorithm 1 gives the decay and the
 * process noise the shape (N, D), time-invariant: abar[n,d], pbar[n,d] per head,
 * [H, dk, dv].  The recursion is the same with abar_t[n] -> abar[h,n,d]; the
 * gate gradients are then sums over (b, t), returned per (b, h) (summed over t)
 * together with the sum over t of the absolute values of up to three linear
 * combinations c_a dabar_t + c_p dpbar_t of the per-token terms (the caller's
 * coefficients, [3][H, dk, dv]): the scale against which the rounding of such
 * sums is measured.
 */
#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

typedef struct {
    int B, T, H, dk, dv;
    const double *q, *k, *v, *a, *p, *r;
    const double *lam0, *eta0;
    double *y, *yvar, *lamT, *etaT;
    /* backward only */
    const double *dy, *dyvar, *dlamT, *detaT;
    double *dq, *dk_, *dv_, *da, *dp, *dr, *dlam0, *deta0;
    /* gates per (n, d): abar, pbar [H, dk, dv]; sums over t of the gate gradients and of
       |ca[j] dabar_t + cp[j] dpbar_t|, per (b, h): ga, gp [B, H, dk, dv], mass [3][B, H, dk, dv] */
    int gate_nd;
    const double *ca, *cp;
    double *ga, *gp, *mass;
    /* work distribution */
    int next;                 /* next (b,h) pair to take */
    pthread_mutex_t lock;
} job_t;

static size_t tok(const job_t* J, int b, int t, int h, int width) {
    return (((size_t)b * J->T + t) * J->H + h) * (size_t)width;
}
static size_t bel(const job_t* J, int b, int h) {
    return ((size_t)b * J->H + h) * (size_t)J->dk * J->dv;
}

/* index of the gate of (b, t, h, n, d) */
static size_t gate(const job_t* J, int b, int t, int h, int n, int d) {
    if (J->gate_nd) return ((size_t)h * J->dk + n) * J->dv + d;
    return tok(J, b, t, h, J->dk) + n;
}

static int take(job_t* J) {
    pthread_mutex_lock(&J->lock);
    int i = J->next < J->B * J->H ? J->next++ : -1;
    pthread_mutex_unlock(&J->lock);
    return i;
}

/* ---------------------------------------------------------------- forward */

static void forward_pair(const job_t* J, int b, int h, double* lam, double* eta) {
    const int dk = J->dk, dv = J->dv;
    const size_t s0 = bel(J, b, h);
    for (int i = 0; i < dk * dv; ++i) {
        lam[i] = J->lam0 ? J->lam0[s0 + i] : 1.0;   /* default prior precision 1 */
        eta[i] = J->eta0 ? J->eta0[s0 + i] : 0.0;   /* default prior mean 0 */
    }
    for (int t = 0; t < J->T; ++t) {
        const double* qt = J->q + tok(J, b, t, h, dk);
        const double* kt = J->k + tok(J, b, t, h, dk);
        const double* at = J->gate_nd ? NULL : J->a + tok(J, b, t, h, dk);
        const double* pt = J->gate_nd ? NULL : J->p + tok(J, b, t, h, dk);
        const double* vt = J->v + tok(J, b, t, h, dv);
        const double* rt = J->r + tok(J, b, t, h, dv);
        double* yt = J->y ? J->y + tok(J, b, t, h, dv) : NULL;
        double* wt = J->yvar ? J->yvar + tok(J, b, t, h, dv) : NULL;
        for (int d = 0; d < dv; ++d) {
            if (yt) yt[d] = 0.0;
            if (wt) wt[d] = 0.0;
        }
        for (int n = 0; n < dk; ++n) {
            for (int d = 0; d < dv; ++d) {
                double* L = &lam[n * dv + d];
                double* E = &eta[n * dv + d];
                const size_t ig = gate(J, b, t, h, n, d);
                const double an = J->gate_nd ? J->a[ig] : at[n], pn = J->gate_nd ? J->p[ig] : pt[n];
                /* predict + update, Theorem 1 (gate view) and Theorem 2 */
                double rho = 1.0 / (an * an + pn * (*L));
                double f = an * rho;
                *L = rho * (*L) + kt[n] * kt[n] * rt[d];
                *E = f * (*E) + kt[n] * rt[d] * vt[d];
                /* readout of the posterior mean (and variance) with the query */
                double inv = 1.0 / (*L);
                if (yt) yt[d] += qt[n] * (*E) * inv;
                if (wt) wt[d] += qt[n] * qt[n] * inv;
            }
        }
    }
    if (J->lamT) memcpy(J->lamT + s0, lam, sizeof(double) * dk * dv);
    if (J->etaT) memcpy(J->etaT + s0, eta, sizeof(double) * dk * dv);
}

static void* forward_worker(void* arg) {
    job_t* J = (job_t*)arg;
    size_t n = (size_t)J->dk * J->dv;
    double* lam = (double*)malloc(sizeof(double) * n);
    double* eta = (double*)malloc(sizeof(double) * n);
    for (int i; (i = take(J)) >= 0;) forward_pair(J, i / J->H, i % J->H, lam, eta);
    free(lam);
    free(eta);
    return NULL;
}

/* --------------------------------------------------------------- backward */

/* Reverse mode of one scalar filter (b, h, n, d).  lt/et hold the trajectory:
 * index 0 is the prior belief, index t is the posterior after token t. */
static void backward_filter(const job_t* J, int b, int h, int n, int d, double* lt, double* et) {
    const int T = J->T, dk = J->dk, dv = J->dv;
    const size_t s0 = bel(J, b, h) + (size_t)n * dv + d;
    lt[0] = J->lam0 ? J->lam0[s0] : 1.0;
    et[0] = J->eta0 ? J->eta0[s0] : 0.0;
    for (int t = 0; t < T; ++t) {
        size_t ik = tok(J, b, t, h, dk) + n, iv = tok(J, b, t, h, dv) + d, ig = gate(J, b, t, h, n, d);
        double a = J->a[ig], p = J->p[ig], k = J->k[ik], r = J->r[iv], v = J->v[iv];
        double rho = 1.0 / (a * a + p * lt[t]);
        lt[t + 1] = rho * lt[t] + k * k * r;
        et[t + 1] = a * rho * et[t] + k * r * v;
    }
    double gl = J->dlamT ? J->dlamT[s0] : 0.0;   /* adjoint of lam_t */
    double ge = J->detaT ? J->detaT[s0] : 0.0;   /* adjoint of eta_t */
    double sa = 0.0, sp = 0.0, sm[3] = {0.0, 0.0, 0.0};   /* gates per (n, d): sums over t */
    for (int t = T - 1; t >= 0; --t) {
        size_t ik = tok(J, b, t, h, dk) + n, iv = tok(J, b, t, h, dv) + d, ig = gate(J, b, t, h, n, d);
        double a = J->a[ig], p = J->p[ig], k = J->k[ik], q = J->q[ik];
        double r = J->r[iv], v = J->v[iv], g = J->dy[iv];
        double lp = lt[t], ep = et[t], lc = lt[t + 1], ec = et[t + 1];
        /* readout y_t[d] += q * eta / lam */
        double mu = ec / lc;
        J->dq[ik] += mu * g;
        double dmu = q * g;
        ge += dmu / lc;
        gl -= dmu * ec / (lc * lc);
        /* readout variance yvar_t[d] += q^2 / lam */
        if (J->dyvar) {
            double gv = J->dyvar[iv];
            J->dq[ik] += 2.0 * q * gv / lc;
            gl -= q * q * gv / (lc * lc);
        }
        /* eta_t = f * eta_{t-1} + k r v,  f = a * rho */
        double den = a * a + p * lp, rho = 1.0 / den, f = a * rho;
        double df = ge * ep;
        J->dk_[ik] += ge * r * v;
        J->dr[iv] += ge * k * v;
        J->dv_[iv] += ge * k * r;
        double ge_prev = f * ge;
        double dat = df * rho;   /* this token's gradients of abar and pbar */
        double drho = df * a;
        /* lam_t = rho * lam_{t-1} + k^2 r */
        drho += gl * lp;
        double gl_prev = gl * rho;
        J->dk_[ik] += gl * 2.0 * k * r;
        J->dr[iv] += gl * k * k;
        /* rho = 1 / (a^2 + p lam_{t-1}) */
        double dden = -drho * rho * rho;
        dat += dden * 2.0 * a;
        double dpt = dden * lp;
        if (J->gate_nd) {
            sa += dat;
            sp += dpt;
            for (int j = 0; j < 3; ++j) sm[j] += fabs(J->ca[j * (size_t)J->H * dk * dv + ig] * dat +
                                                      J->cp[j * (size_t)J->H * dk * dv + ig] * dpt);
        } else {
            J->da[ik] += dat;
            J->dp[ik] += dpt;
        }
        gl_prev += dden * p;
        gl = gl_prev;
        ge = ge_prev;
    }
    if (J->dlam0) J->dlam0[s0] = gl;
    if (J->deta0) J->deta0[s0] = ge;
    if (J->gate_nd) {
        const size_t nb = (size_t)J->B * J->H * dk * dv;
        J->ga[s0] = sa;
        J->gp[s0] = sp;
        for (int j = 0; j < 3; ++j) J->mass[j * nb + s0] = sm[j];
    }
}

static void* backward_worker(void* arg) {
    job_t* J = (job_t*)arg;
    double* lt = (double*)malloc(sizeof(double) * (J->T + 1));
    double* et = (double*)malloc(sizeof(double) * (J->T + 1));
    for (int i; (i = take(J)) >= 0;)
        for (int n = 0; n < J->dk; ++n)
            for (int d = 0; d < J->dv; ++d) backward_filter(J, i / J->H, i % J->H, n, d, lt, et);
    free(lt);
    free(et);
    return NULL;
}

static void run(job_t* J, void* (*fn)(void*), int nthreads) {
    if (nthreads <= 0) nthreads = (int)sysconf(_SC_NPROCESSORS_ONLN);
    if (nthreads > J->B * J->H) nthreads = J->B * J->H;
    if (nthreads < 1) nthreads = 1;
    J->next = 0;
    pthread_mutex_init(&J->lock, NULL);
    pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * nthreads);
    for (int i = 0; i < nthreads; ++i) pthread_create(&th[i], NULL, fn, J);
    for (int i = 0; i < nthreads; ++i) pthread_join(th[i], NULL);
    free(th);
    pthread_mutex_destroy(&J->lock);
}

/* ------------------------------------------------------------- public API */

/* y, yvar, lamT, etaT may each be NULL; lam0 / eta0 NULL mean 1 / 0. */
void kla_oracle_forward(int B, int T, int H, int dk, int dv,
                        const double* q, const double* k, const double* v,
                        const double* a, const double* p, const double* r,
                        const double* lam0, const double* eta0,
                        double* y, double* yvar, double* lamT, double* etaT, int nthreads) {
    job_t J;
    memset(&J, 0, sizeof J);
    J.B = B; J.T = T; J.H = H; J.dk = dk; J.dv = dv;
    J.q = q; J.k = k; J.v = v; J.a = a; J.p = p; J.r = r;
    J.lam0 = lam0; J.eta0 = eta0; J.y = y; J.yvar = yvar; J.lamT = lamT; J.etaT = etaT;
    run(&J, forward_worker, nthreads);
}

/* Gradients are written (not accumulated) into dq..dr, dlam0, deta0; dyvar
 * (upstream gradient of yvar, [B, T, H, dv]), dlamT and detaT NULL mean zero;
 * dlam0 / deta0 may be NULL. */
void kla_oracle_backward(int B, int T, int H, int dk, int dv,
                         const double* q, const double* k, const double* v,
                         const double* a, const double* p, const double* r,
                         const double* lam0, const double* eta0,
                         const double* dy, const double* dyvar, const double* dlamT, const double* detaT,
                         double* dq, double* dk_, double* dv_, double* da, double* dp, double* dr,
                         double* dlam0, double* deta0, int nthreads) {
    job_t J;
    memset(&J, 0, sizeof J);
    J.B = B; J.T = T; J.H = H; J.dk = dk; J.dv = dv;
    J.q = q; J.k = k; J.v = v; J.a = a; J.p = p; J.r = r;
    J.lam0 = lam0; J.eta0 = eta0; J.dy = dy; J.dyvar = dyvar; J.dlamT = dlamT; J.detaT = detaT;
    J.dq = dq; J.dk_ = dk_; J.dv_ = dv_; J.da = da; J.dp = dp; J.dr = dr;
    J.dlam0 = dlam0; J.deta0 = deta0;
    size_t nk = (size_t)B * T * H * dk, nv = (size_t)B * T * H * dv;
    memset(dq, 0, sizeof(double) * nk);
    memset(dk_, 0, sizeof(double) * nk);
    memset(da, 0, sizeof(double) * nk);
    memset(dp, 0, sizeof(double) * nk);
    memset(dv_, 0, sizeof(double) * nv);
    memset(dr, 0, sizeof(double) * nv);
    run(&J, backward_worker, nthreads);
}

/* The forward with gates per (n, d): a, p [H, dk, dv], time-invariant. */
void kla_oracle_forward_nd(int B, int T, int H, int dk, int dv,
                           const double* q, const double* k, const double* v,
                           const double* a, const double* p, const double* r,
                           const double* lam0, const double* eta0,
                           double* y, double* yvar, double* lamT, double* etaT, int nthreads) {
    job_t J;
    memset(&J, 0, sizeof J);
    J.B = B; J.T = T; J.H = H; J.dk = dk; J.dv = dv; J.gate_nd = 1;
    J.q = q; J.k = k; J.v = v; J.a = a; J.p = p; J.r = r;
    J.lam0 = lam0; J.eta0 = eta0; J.y = y; J.yvar = yvar; J.lamT = lamT; J.etaT = etaT;
    run(&J, forward_worker, nthreads);
}

/* The backward with gates per (n, d): dq, dk, dv, dr, dlam0, deta0 as in
 * kla_oracle_backward; ga, gp [B, H, dk, dv] receive the sums over t of the gradients
 * of abar and pbar, mass [3][B, H, dk, dv] the sums over t of
 * |ca[j] dabar_t + cp[j] dpbar_t| (ca, cp [3][H, dk, dv]). */
void kla_oracle_backward_nd(int B, int T, int H, int dk, int dv,
                            const double* q, const double* k, const double* v,
                            const double* a, const double* p, const double* r,
                            const double* lam0, const double* eta0,
                            const double* dy, const double* dyvar, const double* dlamT, const double* detaT,
                            double* dq, double* dk_, double* dv_, double* dr, double* dlam0, double* deta0,
                            const double* ca, const double* cp, double* ga, double* gp, double* mass,
                            int nthreads) {
    job_t J;
    memset(&J, 0, sizeof J);
    J.B = B; J.T = T; J.H = H; J.dk = dk; J.dv = dv; J.gate_nd = 1;
    J.q = q; J.k = k; J.v = v; J.a = a; J.p = p; J.r = r;
    J.lam0 = lam0; J.eta0 = eta0; J.dy = dy; J.dyvar = dyvar; J.dlamT = dlamT; J.detaT = detaT;
    J.dq = dq; J.dk_ = dk_; J.dv_ = dv_; J.dr = dr; J.dlam0 = dlam0; J.deta0 = deta0;
    J.ca = ca; J.cp = cp; J.ga = ga; J.gp = gp; J.mass = mass;
    size_t nk = (size_t)B * T * H * dk, nv = (size_t)B * T * H * dv;
    memset(dq, 0, sizeof(double) * nk);
    memset(dk_, 0, sizeof(double) * nk);
    memset(dv_, 0, sizeof(double) * nv);
    memset(dr, 0, sizeof(double) * nv);
    run(&J, backward_worker, nthreads);
}

/* One recurrent step on a carried belief, updated in place (the O(1) per token
 * inference form): inputs [S, H, *], lam / eta [S, H, dk, dv]. */
void kla_oracle_decode_step(int S, int H, int dk, int dv,
                            const double* q, const double* k, const double* v,
                            const double* a, const double* p, const double* r,
                            double* lam, double* eta, double* y, double* yvar) {
    job_t J;
    memset(&J, 0, sizeof J);
    J.B = S; J.T = 1; J.H = H; J.dk = dk; J.dv = dv;
    J.q = q; J.k = k; J.v = v; J.a = a; J.p = p; J.r = r;
    J.y = y; J.yvar = yvar;
    size_t n = (size_t)dk * dv;
    double* L = (double*)malloc(sizeof(double) * n);
    double* E = (double*)malloc(sizeof(double) * n);
    for (int s = 0; s < S; ++s)
        for (int h = 0; h < H; ++h) {
            size_t s0 = bel(&J, s, h);
            J.lam0 = lam; J.eta0 = eta; J.lamT = NULL; J.etaT = NULL;
            forward_pair(&J, s, h, L, E);
            memcpy(lam + s0, L, sizeof(double) * n);
            memcpy(eta + s0, E, sizeof(double) * n);
        }
    free(L);
    free(E);
}

/* Full trajectory of one sequence (B = H = 1): lam_traj / eta_traj [T+1, dk, dv],
 * row 0 the prior belief.  Used by the tests that compare the recursion with
 * scans and closed forms. */
void kla_oracle_trace(int T, int dk, int dv,
                      const double* k, const double* v, const double* a, const double* p,
                      const double* r, const double* lam0, const double* eta0,
                      double* lam_traj, double* eta_traj) {
    size_t n = (size_t)dk * dv;
    for (size_t i = 0; i < n; ++i) {
        lam_traj[i] = lam0 ? lam0[i] : 1.0;
        eta_traj[i] = eta0 ? eta0[i] : 0.0;
    }
    for (int t = 0; t < T; ++t) {
        const double *L = lam_traj + t * n, *E = eta_traj + t * n;
        double *L1 = lam_traj + (t + 1) * n, *E1 = eta_traj + (t + 1) * n;
        for (int i = 0; i < dk; ++i)
            for (int d = 0; d < dv; ++d) {
                size_t j = (size_t)i * dv + d;
                double ai = a[t * dk + i], pi = p[t * dk + i], ki = k[t * dk + i];
                double rd = r[t * dv + d], vd = v[t * dv + d];
                double rho = 1.0 / (ai * ai + pi * L[j]);
                L1[j] = rho * L[j] + ki * ki * rd;
                E1[j] = ai * rho * E[j] + ki * rd * vd;
            }
    }
}

/* ---- the two associative operators of Corollaries 1 and 2 (scalar lanes) ---- */

/* Theorem 1: the per-token Moebius matrix [[alpha, beta], [gamma, delta]]. */
void kla_oracle_mobius_matrix(double k, double a, double p, double r, double M[4]) {
    double phi = k * k * r;
    M[0] = 1.0 + p * phi;   /* alpha */
    M[1] = a * a * phi;     /* beta  */
    M[2] = p;               /* gamma */
    M[3] = a * a;           /* delta */
}

/* Composition "M2 after M1" is the matrix product M2 * M1 (Corollary 1). */
void kla_oracle_mobius_compose(const double M2[4], const double M1[4], double out[4]) {
    double o0 = M2[0] * M1[0] + M2[1] * M1[2];
    double o1 = M2[0] * M1[1] + M2[1] * M1[3];
    double o2 = M2[2] * M1[0] + M2[3] * M1[2];
    double o3 = M2[2] * M1[1] + M2[3] * M1[3];
    out[0] = o0; out[1] = o1; out[2] = o2; out[3] = o3;
}

/* Action of a Moebius matrix on a precision: (alpha l + beta) / (gamma l + delta). */
double kla_oracle_mobius_apply(const double M[4], double lam) {
    return (M[0] * lam + M[1]) / (M[2] * lam + M[3]);
}

/* Corollary 2: (f2, b2) o (f1, b1) = (f2 f1, f2 b1 + b2), elementwise over m lanes. */
void kla_oracle_affine_compose(int m, const double* f2, const double* b2,
                               const double* f1, const double* b1, double* fo, double* bo) {
    for (int i = 0; i < m; ++i) {
        double f = f2[i] * f1[i], b = f2[i] * b1[i] + b2[i];
        fo[i] = f;
        bo[i] = b;
    }
}
