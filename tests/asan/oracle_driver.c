/* Host sanitizer run of the fp64 oracle (built with -fsanitize=address,undefined):
 * every public entry point on small shapes, with optional arguments both given and
 * NULL, several thread counts, and a check that the outputs are finite.  Exit 0 on
 * success; the sanitizers abort on any invalid access. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

void kla_oracle_forward(int B, int T, int H, int dk, int dv, const double* q, const double* k, const double* v,
                        const double* a, const double* p, const double* r, const double* lam0, const double* eta0,
                        double* y, double* yvar, double* lamT, double* etaT, int nthreads);
void kla_oracle_backward(int B, int T, int H, int dk, int dv, const double* q, const double* k, const double* v,
                         const double* a, const double* p, const double* r, const double* lam0, const double* eta0,
                         const double* dy, const double* dyvar, const double* dlamT, const double* detaT,
                         double* dq, double* dk_, double* dv_, double* da, double* dp, double* dr, double* dlam0,
                         double* deta0, int nthreads);
void kla_oracle_forward_nd(int B, int T, int H, int dk, int dv, const double* q, const double* k, const double* v,
                           const double* a, const double* p, const double* r, const double* lam0,
                           const double* eta0, double* y, double* yvar, double* lamT, double* etaT, int nthreads);
void kla_oracle_backward_nd(int B, int T, int H, int dk, int dv, const double* q, const double* k, const double* v,
                            const double* a, const double* p, const double* r, const double* lam0,
                            const double* eta0, const double* dy, const double* dyvar, const double* dlamT,
                            const double* detaT, double* dq, double* dk_, double* dv_, double* dr, double* dlam0,
                            double* deta0, const double* ca, const double* cp, double* ga, double* gp, double* mass,
                            int nthreads);
void kla_oracle_decode_step(int S, int H, int dk, int dv, const double* q, const double* k, const double* v,
                            const double* a, const double* p, const double* r, double* lam, double* eta, double* y,
                            double* yvar);
void kla_oracle_mobius_matrix(double k, double a, double p, double r, double M[4]);
void kla_oracle_mobius_compose(const double M2[4], const double M1[4], double out[4]);
double kla_oracle_mobius_apply(const double M[4], double lam);

static unsigned long long st = 88172645463325252ull;
static double unif(void) {   /* xorshift64 */
    st ^= st << 13;
    st ^= st >> 7;
    st ^= st << 17;
    return (double)(st >> 11) * 0x1p-53;
}
static double* arr(size_t n, double lo, double hi) {
    double* x = malloc(n * sizeof(double));
    for (size_t i = 0; i < n; ++i) x[i] = lo + (hi - lo) * unif();
    return x;
}
static double* out(size_t n) { return calloc(n, sizeof(double)); }
static int finite(const double* x, size_t n) {
    for (size_t i = 0; i < n; ++i)
        if (!isfinite(x[i])) return 0;
    return 1;
}
#define CHECK(c)                                                  \
    do {                                                          \
        if (!(c)) {                                               \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            return 1;                                             \
        }                                                         \
    } while (0)

static int run_shape(int B, int T, int H, int dk, int dv, int nthreads) {
    const size_t nk = (size_t)B * T * H * dk, nv = (size_t)B * T * H * dv, nb = (size_t)B * H * dk,
                 ne = (size_t)B * H * dk * dv, ng = (size_t)H * dk * dv, nt = (size_t)B * T * H;
    double *q = arr(nk, -1, 1), *k = arr(nk, -1, 1), *v = arr(nv, -1, 1), *a = arr(nk, 0.3, 1.0),
           *p = arr(nk, 0.0, 0.5), *r = arr(nv, 0.2, 1.2), *lam0 = arr(ne, 0.5, 1.5), *eta0 = arr(ne, -1, 1);
    double *an = arr(ng, 0.3, 1.0), *pn = arr(ng, 0.0, 0.5), *ca = arr(3 * ng, -1, 1), *cp = arr(3 * ng, -1, 1);
    double *dy = arr(nv, -1, 1), *dyvar = arr(nv, -1, 1), *dlamT = arr(ne, -1, 1), *detaT = arr(ne, -1, 1);
    double *y = out(nv), *yvar = out(nv), *lamT = out(ne), *etaT = out(ne);
    double *dq = out(nk), *dk_ = out(nk), *dv_ = out(nv), *da = out(nk), *dp = out(nk), *dr = out(nv),
           *dlam0 = out(ne), *deta0 = out(ne), *ga = out(ne), *gp = out(ne), *mass = out(3 * ne);
    (void)nb;
    (void)nt;
    kla_oracle_forward(B, T, H, dk, dv, q, k, v, a, p, r, lam0, eta0, y, yvar, lamT, etaT, nthreads);
    CHECK(finite(y, nv) && finite(yvar, nv) && finite(lamT, ne) && finite(etaT, ne));
    kla_oracle_forward(B, T, H, dk, dv, q, k, v, a, p, r, NULL, NULL, y, NULL, NULL, NULL, nthreads);
    CHECK(finite(y, nv));
    kla_oracle_backward(B, T, H, dk, dv, q, k, v, a, p, r, lam0, eta0, dy, dyvar, dlamT, detaT, dq, dk_, dv_, da,
                        dp, dr, dlam0, deta0, nthreads);
    CHECK(finite(dq, nk) && finite(dk_, nk) && finite(dv_, nv) && finite(da, nk) && finite(dp, nk) &&
          finite(dr, nv) && finite(dlam0, ne) && finite(deta0, ne));
    kla_oracle_backward(B, T, H, dk, dv, q, k, v, a, p, r, NULL, NULL, dy, NULL, NULL, NULL, dq, dk_, dv_, da, dp,
                        dr, NULL, NULL, nthreads);
    CHECK(finite(dq, nk) && finite(dr, nv));
    kla_oracle_forward_nd(B, T, H, dk, dv, q, k, v, an, pn, r, lam0, eta0, y, yvar, lamT, etaT, nthreads);
    CHECK(finite(y, nv) && finite(etaT, ne));
    kla_oracle_backward_nd(B, T, H, dk, dv, q, k, v, an, pn, r, lam0, eta0, dy, dyvar, dlamT, detaT, dq, dk_, dv_,
                           dr, dlam0, deta0, ca, cp, ga, gp, mass, nthreads);
    CHECK(finite(ga, ne) && finite(gp, ne) && finite(mass, 3 * ne) && finite(deta0, ne));
    /* decode: S = B sequences, one token, belief in place */
    {
        const size_t sk = (size_t)B * H * dk, sv = (size_t)B * H * dv;
        double *lam = arr(ne, 0.5, 1.5), *eta = arr(ne, -1, 1), *yd = out(sv), *yvd = out(sv);
        double *qs = arr(sk, -1, 1), *ks = arr(sk, -1, 1), *as = arr(sk, 0.3, 1.0), *ps = arr(sk, 0.0, 0.5);
        double *vs = arr(sv, -1, 1), *rs = arr(sv, 0.2, 1.2);
        kla_oracle_decode_step(B, H, dk, dv, qs, ks, vs, as, ps, rs, lam, eta, yd, yvd);
        CHECK(finite(lam, ne) && finite(eta, ne) && finite(yd, sv) && finite(yvd, sv));
        double* dall[] = {lam, eta, yd, yvd, qs, ks, as, ps, vs, rs};
        for (size_t i = 0; i < sizeof dall / sizeof dall[0]; ++i) free(dall[i]);
    }
    double M1[4], M2[4], M[4];
    kla_oracle_mobius_matrix(0.5, 0.9, 0.1, 0.7, M1);
    kla_oracle_mobius_matrix(-0.3, 0.8, 0.2, 1.1, M2);
    kla_oracle_mobius_compose(M2, M1, M);
    CHECK(isfinite(kla_oracle_mobius_apply(M, 1.3)));
    double* all[] = {q, k, v, a, p, r, lam0, eta0, an, pn, ca, cp, dy, dyvar, dlamT, detaT, y, yvar, lamT, etaT,
                     dq, dk_, dv_, da, dp, dr, dlam0, deta0, ga, gp, mass};
    for (size_t i = 0; i < sizeof all / sizeof all[0]; ++i) free(all[i]);
    return 0;
}

int main(void) {
    int rc = 0;
    rc |= run_shape(2, 9, 2, 3, 4, 1);
    rc |= run_shape(1, 1, 1, 1, 1, 3);
    rc |= run_shape(3, 17, 2, 5, 2, 4);
    rc |= run_shape(1, 0, 2, 2, 2, 2);
    if (rc == 0) printf("oracle sanitizer run: ok\n");
    return rc;
}
