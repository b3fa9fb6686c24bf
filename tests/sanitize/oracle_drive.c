/* Drives every function of the CPU oracle (oracle/finc_oracle.c) on small,
 * ragged and empty shapes, for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer: every buffer is allocated at exactly the size
 * the function's documented layout gives, so a read or write past it stops
 * the run.  Return codes must be 0 (the checks of values live in the pins).
 * Test infrastructure: built and run by tests/test_sanitizers_cpu.py. */
#include <stdio.h>
#include <stdlib.h>

int orc_forward(const double *, double *, const double *, long, int, int, int, int, int);
int orc_inverse(const double *, double *, const double *, long, int, int, int, int, int);
int orc_logdet(const double *, int, int, int, int, int, double *);
int orc_backward(const double *, const double *, const double *, double *, double *, double,
                 long, int, int, int, int, int);
int orc_unit_forward(const double *, double *, const double *, long, int, int, int, int);
int orc_unit_inverse(const double *, double *, const double *, long, int, int, int, int);
int orc_unit_logdet(const double *, int, int, int, int, double *);
int orc_unit_backward(const double *, const double *, const double *, double *, double *, double,
                      long, int, int, int, int);
int orc_split_forward(const double *, double *, const double *, long, int, int, int, int);
int orc_split_inverse(const double *, double *, const double *, long, int, int, int, int);
int orc_split_logdet(const double *, int, int, int, int, double *);
int orc_split_backward(const double *, const double *, const double *, double *, double *, double,
                       long, int, int, int, int);
void orc_actnorm_forward(const double *, double *, const double *, const double *, long, int, int,
                         int);
void orc_actnorm_inverse(const double *, double *, const double *, const double *, long, int, int,
                         int);
int orc_actnorm_backward(const double *, const double *, const double *, double *, double *,
                         double *, double, long, int, int, int);
void orc_squeeze(const double *, double *, long, int, int, int);
void orc_unsqueeze(const double *, double *, long, int, int, int);
int orc_stack_forward(const double *, double *const *, const double *, const double *,
                      const double *, long, int, int, int, int, int, int);
int orc_stack_inverse(const double *const *, double *, const double *, const double *,
                      const double *, long, int, int, int, int, int, int);
int orc_stack_logdet(const double *, const double *, int, int, int, int, int, int, double *);
int orc_stack_backward(const double *, const double *const *, const double *, const double *,
                       const double *, double *, double *, double *, double *, double, long, int,
                       int, int, int, int, int);
int orc_gauss_nll(const double *const *, const long *, int, long, const double *, double *,
                  double *);
int orc_conv1x1_forward(const double *, double *, const double *, long, int, int, int);
int orc_conv1x1_inverse(const double *, double *, const double *, long, int, int, int);
int orc_conv1x1_logdet(const double *, int, int, int, double *);
int orc_coupling_net(const double *, double *, const double *, long, int, int, int, int);
int orc_coupling_forward(const double *, double *, const double *, long, int, int, int, int,
                         double *);
int orc_coupling_inverse(const double *, double *, const double *, long, int, int, int, int);
int orc_step_forward(const double *, double *, const double *, long, int, int, int, int, int,
                     double *);
int orc_step_inverse(const double *, double *, const double *, long, int, int, int, int, int);
long orc_flow_params(int, int, int, int, int);
int orc_flow_forward(const double *, double *const *, const double *, long, int, int, int, int,
                     int, int, int, double *);
int orc_flow_sample(const double *const *, double *, const double *, long, int, int, int, int,
                    int, int, int);

static unsigned long long state = 88172645463325252ull;
static double uni(void) {   /* xorshift64, values in [-1, 1) */
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return (double)(state >> 11) / 4503599627370496.0 - 1.0;
}
static double *arr(long n) {   /* exactly n doubles (malloc(0) for none) */
    double *p = malloc(sizeof(double) * (size_t)n);
    for (long i = 0; i < n; ++i)
        p[i] = uni();
    return p;
}
/* Weights with every diagonal entry of magnitude >= 0.5, so inverses exist. */
static double *kernel(int nblk, int C, int k) {
    double *K = arr((long)nblk * C * C * k * k);
    for (int q = 0; q < nblk; ++q)
        for (int c = 0; c < C; ++c)
            for (int t = 0; t < k * k; ++t) {
                double *v = &K[(((long)q * C + c) * C + c) * k * k + t];
                *v = *v < 0 ? *v - 0.5 : *v + 0.5;
            }
    return K;
}

static int failures = 0;
#define CHECK(call)                                                       \
    do {                                                                  \
        int rc_ = (call);                                                 \
        if (rc_ != 0) {                                                   \
            fprintf(stderr, "%s:%d: %s returned %d\n", __FILE__, __LINE__, #call, rc_); \
            ++failures;                                                   \
        }                                                                 \
    } while (0)

static void layer_and_units(long B, int C, int H, int W, int k) {
    const long n = B * C * H * W;
    double *x = arr(n), *y = arr(n), *dy = arr(n), *dx = arr(n), ld;
    for (int corner = 0; corner < 4; ++corner) {
        double *K = kernel(1, C, k), *dK = arr((long)C * C * k * k);
        CHECK(orc_forward(x, y, K, B, C, H, W, k, corner));
        CHECK(orc_inverse(y, dx, K, B, C, H, W, k, corner));
        CHECK(orc_logdet(K, C, k, corner, H, W, &ld));
        CHECK(orc_backward(x, dy, K, dx, dK, -1.0, B, C, H, W, k, corner));
        free(K);
        free(dK);
    }
    double *K4 = kernel(4, C, k), *dK4 = arr(4L * C * C * k * k);
    CHECK(orc_unit_forward(x, y, K4, B, C, H, W, k));
    CHECK(orc_unit_inverse(y, dx, K4, B, C, H, W, k));
    CHECK(orc_unit_logdet(K4, C, k, H, W, &ld));
    CHECK(orc_unit_backward(x, dy, K4, dx, dK4, 0.5, B, C, H, W, k));
    double *s = arr(C), *b = arr(C), *ds = arr(C), *db = arr(C);
    for (int c = 0; c < C; ++c)
        s[c] = s[c] < 0 ? s[c] - 0.5 : s[c] + 0.5;
    orc_actnorm_forward(x, y, s, b, B, C, H, W);
    orc_actnorm_inverse(y, dx, s, b, B, C, H, W);
    CHECK(orc_actnorm_backward(x, dy, s, dx, ds, db, -1.0, B, C, H, W));
    double *Wm = kernel(1, C, 1);
    CHECK(orc_conv1x1_forward(x, y, Wm, B, C, H, W));
    CHECK(orc_conv1x1_inverse(y, dx, Wm, B, C, H, W));
    CHECK(orc_conv1x1_logdet(Wm, C, H, W, &ld));
    if (C % 4 == 0) {
        const int q = C / 4;
        double *Kq4 = kernel(4, q, k), *dKq4 = arr(4L * q * q * k * k);
        CHECK(orc_split_forward(x, y, Kq4, B, C, H, W, k));
        CHECK(orc_split_inverse(y, dx, Kq4, B, C, H, W, k));
        CHECK(orc_split_logdet(Kq4, C, k, H, W, &ld));
        CHECK(orc_split_backward(x, dy, Kq4, dx, dKq4, 0.25, B, C, H, W, k));
        free(Kq4);
        free(dKq4);
    }
    if (H % 2 == 0 && W % 2 == 0) {
        double *sq = arr(n);
        orc_squeeze(x, sq, B, C, H, W);
        orc_unsqueeze(sq, y, B, 4 * C, H / 2, W / 2);
        free(sq);
    }
    free(x); free(y); free(dy); free(dx); free(K4); free(dK4);
    free(s); free(b); free(ds); free(db); free(Wm);
}

static void stack(long B, int L, int U, int C1, int H1, int W1, int k) {
    long nK = 0, nS = 0;
    for (int l = 0; l < L; ++l) {
        const long C = (long)C1 << l;
        nK += (long)U * 4 * C * C * k * k;
        nS += (long)U * C;
    }
    double *K = arr(nK), *sc = arr(nS), *bi = arr(nS), *x = arr(B * C1 * H1 * W1), *xr;
    for (long i = 0; i < nS; ++i)
        sc[i] = sc[i] < 0 ? sc[i] - 0.5 : sc[i] + 0.5;
    double *z[8];
    for (int l = 0; l < L; ++l) {
        const long C = (long)C1 << l, hw = (long)(H1 >> l) * (W1 >> l);
        z[l] = arr(B * (l < L - 1 ? C / 2 : C) * hw);
    }
    /* keep the kernels' diagonals away from 0 level by level */
    long off = 0;
    for (int l = 0; l < L; ++l) {
        const int C = C1 << l;
        for (int u = 0; u < 4 * U; ++u, off += (long)C * C * k * k)
            for (int c = 0; c < C; ++c)
                for (int t = 0; t < k * k; ++t) {
                    double *v = &K[off + ((long)c * C + c) * k * k + t];
                    *v = *v < 0 ? *v - 0.5 : *v + 0.5;
                }
    }
    xr = arr(B * C1 * H1 * W1);
    CHECK(orc_stack_forward(x, z, K, sc, bi, B, L, U, C1, H1, W1, k));
    CHECK(orc_stack_inverse((const double *const *)z, xr, K, sc, bi, B, L, U, C1, H1, W1, k));
    double ld, *dx = arr(B * C1 * H1 * W1), *dK = arr(nK), *ds = arr(nS), *db = arr(nS);
    CHECK(orc_stack_logdet(K, sc, L, U, C1, H1, W1, k, &ld));
    CHECK(orc_stack_backward(x, (const double *const *)z, K, sc, bi, dx, dK, ds, db, -1.0, B, L,
                             U, C1, H1, W1, k));
    free(dx); free(dK); free(ds); free(db);
    for (int l = 0; l < L; ++l)
        free(z[l]);
    free(K); free(sc); free(bi); free(x); free(xr);
}

static long step_count(int C, int k, int hid) {
    const long q = C / 4, h = C / 2;
    return 4 * q * q * k * k + 2L * C + (long)C * C + (long)hid * h * 9 + hid +
           (long)hid * hid + hid + (long)C * hid * 9 + 2L * C;
}

static void flow_parts(long B) {
    const int C = 8, H = 3, W = 5, k = 3, hid = 6;
    const long n = B * C * H * W, ncp = step_count(C, k, hid) - (4L * 4 * k * k + 2 * C + C * C);
    double *x = arr(n), *y = arr(n), *xr = arr(n), *hh = arr(B * C * H * W);
    double *cp = arr(ncp), *sp = arr(step_count(C, k, hid)), *ld = arr(B);
    double *xa = arr(B * (C / 2) * H * W);
    CHECK(orc_coupling_net(xa, hh, cp, B, C, H, W, hid));
    CHECK(orc_coupling_forward(x, y, cp, B, C, H, W, hid, ld));
    CHECK(orc_coupling_inverse(y, xr, cp, B, C, H, W, hid));
    CHECK(orc_step_forward(x, y, sp, B, C, H, W, k, hid, ld));
    CHECK(orc_step_inverse(y, xr, sp, B, C, H, W, k, hid));
    free(x); free(y); free(xr); free(hh); free(cp); free(sp); free(ld); free(xa);
    /* multi-scale flow: L = 2 levels of K = 1 step on (B, 1, 8, 8) */
    const int L = 2, Ks = 1, C0 = 1, H0 = 8, W0 = 8;
    const long np = orc_flow_params(L, Ks, C0, k, hid);
    double *params = arr(np), *img = arr(B * C0 * H0 * W0), *back = arr(B * C0 * H0 * W0);
    double *lg = arr(B), *z[2];
    for (int l = 0; l < L; ++l) {
        const long Cl = 4L * C0 << l, hw = (long)(H0 >> (l + 1)) * (W0 >> (l + 1));
        z[l] = arr(B * (l < L - 1 ? Cl / 2 : Cl) * hw);
    }
    CHECK(orc_flow_forward(img, z, params, B, L, Ks, C0, H0, W0, k, hid, lg));
    CHECK(orc_flow_sample((const double *const *)z, back, params, B, L, Ks, C0, H0, W0, k, hid));
    long nz[2];
    for (int l = 0; l < L; ++l) {
        const long Cl = 4L * C0 << l, hw = (long)(H0 >> (l + 1)) * (W0 >> (l + 1));
        nz[l] = (l < L - 1 ? Cl / 2 : Cl) * hw;
    }
    double *nll = arr(B), *bpd = arr(B);
    CHECK(orc_gauss_nll((const double *const *)z, nz, L, B, lg, nll, bpd));
    free(params); free(img); free(back); free(lg); free(z[0]); free(z[1]); free(nll); free(bpd);
}

int main(void) {
    const int shapes[][5] = {{2, 3, 5, 4, 3}, {1, 1, 1, 1, 1}, {0, 2, 3, 3, 2}, {1, 2, 2, 7, 7},
                             {3, 4, 4, 4, 5}, {2, 8, 6, 4, 3}, {1, 4, 1, 1, 1}, {0, 4, 2, 2, 2},
                             {1, 5, 7, 3, 6}, {2, 12, 2, 6, 4}};
    for (unsigned i = 0; i < sizeof(shapes) / sizeof(shapes[0]); ++i)
        layer_and_units(shapes[i][0], shapes[i][1], shapes[i][2], shapes[i][3], shapes[i][4]);
    stack(2, 2, 1, 2, 4, 4, 3);
    stack(1, 1, 2, 3, 3, 5, 2);
    stack(0, 2, 1, 2, 4, 4, 3);
    flow_parts(2);
    flow_parts(0);
    if (failures)
        fprintf(stderr, "%d calls failed\n", failures);
    else
        printf("oracle sanitizer drive: all calls returned 0\n");
    return failures ? 1 : 0;
}
