/*
 * dro_oracle.c -- plain CPU oracle for the Wasserstein-DRO reservation path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header or constant with the GPU library and includes none of its files.
 *
 * What it computes (paper, Appendix A, Prop. A.1 and Sec. 4.2):
 *   Q(eta, x)       = c_p (x - eta)^+ + c_w (eta - x)^+          stochastic cost, Sec. 3.3,
 *                                                                 with L_in folded into eta = r - L_in
 *   phi(eta, x, g)  = max{ Q(eta,0) - g x,  Q(eta,x),  Q(eta,L) - g (L - x) }
 *                                                                 App. A, Step 4 (candidates at 0, at the sample, at L_max)
 *   S[c,k,m]        = sum over the samples x of class c of phi(eta_k, x, lam_m)
 *                                                                 App. A, Step 5 (LP objective) at theta = phi
 *   J[e,c,k,m]      = lam_m eps[e,c] + S[c,k,m] / N_c            App. A, Step 3 (Kantorovich dual) on a grid of gamma
 *   W[e,c,k]        = min over m of J, m* the lowest m attaining it
 *   k*[e,c]         = lowest k <= kmax_c attaining min over k of W     (Prop. 4.2: optimal r on the grid)
 *   j_c             = ceil(c_p N_c / (c_p + c_w)), q_value = j_c-th smallest sample
 *                                                                 Prop. 4.2, generalized inverse
 *   block step      = one reservation update of Block 1 of Alg. 1 under the memory-capacity constraint (Sec. 3.4),
 *                     Gauss-Seidel over classes (a reading: the paper leaves the grid form open)
 *
 * Two evaluations of S are provided:
 *   - dense fp64: every (c,k,m,n) term in double, summed in sample order;
 *   - exact: every term as a 64-bit integer in units of 2^-33 (all inputs are
 *     integers <= 2^15 or binary32 values in [2^-10, 2^7], so each candidate of
 *     phi is an exact multiple of 2^-33 below 2^56), summed in 128-bit integers.
 *     A value-grouped variant multiplies phi(v) by the number of samples equal
 *     to v; integer addition makes it identical to the per-sample sum.
 * J is then a fully specified double expression of the exact S:
 *   J = RN(RN(lam*eps) + RN(RN(S)/N)), round-to-nearest-even, no contraction.
 *
 * Build: gcc -O2 -std=gnu11 -fopenmp -ffp-contract=off -fno-fast-math -fPIC -shared
 *        (the build() function of oracle/__init__.py).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef __int128 i128;

#define FIX_SHIFT 33

int oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

static inline int32_t seg_of(const int32_t *seg, int32_t c) { return seg ? seg[c] : c; }

/* ------------------------------------------------------------ fp64 dense -- */

/* phi in double precision, written term by term from App. A, Step 4. */
double oracle_phi(int32_t eta, int32_t x, int32_t L, float cp, float cw, float lam)
{
    double e = eta, xx = x, LL = L, p = cp, w = cw, g = lam;
    double q_at_x = p * fmax(xx - e, 0.0) + w * fmax(e - xx, 0.0);   /* at the sample */
    double q_at_0 = w * fmax(e, 0.0) - g * xx;                         /* at 0         */
    double q_at_L = p * (LL - e) - g * (LL - xx);                      /* at L_max     */
    double r = q_at_x;
    if (q_at_0 > r) r = q_at_0;
    if (q_at_L > r) r = q_at_L;
    return r;
}

/* S[c*K*M + k*M + m] = sum_n phi(eta_k, x_n, lam_m) over the samples of class c. */
void oracle_S_f64(int32_t C, const int64_t *offsets, const int32_t *seg, const int32_t *xi,
                  const int32_t *L, int32_t K, const int32_t *eta, int32_t M, const float *lam,
                  const float *cp, const float *cw, double *S)
{
    int64_t total = (int64_t)C * K;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t ck = 0; ck < total; ++ck) {
        int32_t c = (int32_t)(ck / K), k = (int32_t)(ck % K);
        int32_t s = seg_of(seg, c);
        for (int32_t m = 0; m < M; ++m) {
            double acc = 0.0;
            for (int64_t n = offsets[s]; n < offsets[s + 1]; ++n)
                acc += oracle_phi(eta[k], xi[n], L[c], cp[c], cw[c], lam[m]);
            S[(int64_t)c * K * M + (int64_t)k * M + m] = acc;
        }
    }
}

/* ---------------------------------------------------------------- exact -- */

/* v * 2^33 as an integer; returns 0 and sets *ok = 0 if v is not an exact
 * multiple of 2^-33 or is too large for the fixed-point range. */
static int64_t to_fix(float v, int *ok)
{
    double d = ldexp((double)v, FIX_SHIFT);
    if (!(fabs(d) < 0x1p52) || d != floor(d)) { *ok = 0; return 0; }
    return (int64_t)d;
}

int oracle_fix_ok(float v)
{
    int ok = 1;
    (void)to_fix(v, &ok);
    return ok;
}

static inline int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

/* phi in units of 2^-33: the three candidates of Step 4, in exact integers. */
static inline int64_t phi_fix(int64_t eta, int64_t x, int64_t L, int64_t CP, int64_t CW, int64_t G)
{
    int64_t q_at_x = CP * max64(x - eta, 0) + CW * max64(eta - x, 0);
    int64_t q_at_0 = CW * max64(eta, 0) - G * x;
    int64_t q_at_L = CP * (L - eta) - G * (L - x);
    return max64(q_at_x, max64(q_at_0, q_at_L));
}

int64_t oracle_phi_fix(int32_t eta, int32_t x, int32_t L, float cp, float cw, float lam)
{
    int ok = 1;
    int64_t CP = to_fix(cp, &ok), CW = to_fix(cw, &ok), G = to_fix(lam, &ok);
    return phi_fix(eta, x, L, CP, CW, G);
}

typedef struct { int32_t *val; int64_t *cnt; int32_t nv; } vgroup;

static int cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* Distinct sample values of a segment and how often each occurs. */
static vgroup group_values(const int32_t *x, int64_t n)
{
    vgroup g = {0, 0, 0};
    int32_t *tmp = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n ? n : 1));
    memcpy(tmp, x, sizeof(int32_t) * (size_t)n);
    qsort(tmp, (size_t)n, sizeof(int32_t), cmp_i32);
    g.val = (int32_t *)malloc(sizeof(int32_t) * (size_t)(n ? n : 1));
    g.cnt = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n ? n : 1));
    for (int64_t i = 0; i < n; ++i) {
        if (g.nv > 0 && g.val[g.nv - 1] == tmp[i]) { g.cnt[g.nv - 1]++; continue; }
        g.val[g.nv] = tmp[i];
        g.cnt[g.nv] = 1;
        g.nv++;
    }
    free(tmp);
    return g;
}

/* Exact S as a signed 128-bit integer in units of 2^-33, split into
 * (hi, lo) = (S >> 64, S mod 2^64).  grouped = 0: one term per sample;
 * grouped = 1: one term per distinct value times its count.
 * Returns 0, or -1 if a coefficient is outside the exact fixed-point range. */
int oracle_S_exact(int32_t C, const int64_t *offsets, const int32_t *seg, const int32_t *xi,
                   const int32_t *L, int32_t K, const int32_t *eta, int32_t M, const float *lam,
                   const float *cp, const float *cw, int grouped, int64_t *S_hi, uint64_t *S_lo)
{
    int ok = 1;
    for (int32_t c = 0; c < C; ++c) { (void)to_fix(cp[c], &ok); (void)to_fix(cw[c], &ok); }
    for (int32_t m = 0; m < M; ++m) (void)to_fix(lam[m], &ok);
    if (!ok) return -1;

    int32_t S = 0;
    for (int32_t c = 0; c < C; ++c) if (seg_of(seg, c) + 1 > S) S = seg_of(seg, c) + 1;
    vgroup *groups = NULL;
    if (grouped) {
        groups = (vgroup *)calloc((size_t)S, sizeof(vgroup));
        for (int32_t s = 0; s < S; ++s)
            groups[s] = group_values(xi + offsets[s], offsets[s + 1] - offsets[s]);
    }
    int64_t total = (int64_t)C * K;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t ck = 0; ck < total; ++ck) {
        int32_t c = (int32_t)(ck / K), k = (int32_t)(ck % K);
        int32_t s = seg_of(seg, c);
        int okl = 1;
        int64_t CP = to_fix(cp[c], &okl), CW = to_fix(cw[c], &okl);
        for (int32_t m = 0; m < M; ++m) {
            int64_t G = to_fix(lam[m], &okl);
            i128 acc = 0;
            if (grouped) {
                const vgroup *g = &groups[s];
                for (int32_t j = 0; j < g->nv; ++j)
                    acc += (i128)g->cnt[j] * (i128)phi_fix(eta[k], g->val[j], L[c], CP, CW, G);
            } else {
                for (int64_t n = offsets[s]; n < offsets[s + 1]; ++n)
                    acc += (i128)phi_fix(eta[k], xi[n], L[c], CP, CW, G);
            }
            int64_t idx = (int64_t)c * K * M + (int64_t)k * M + m;
            S_hi[idx] = (int64_t)(acc >> 64);
            S_lo[idx] = (uint64_t)acc;
        }
    }
    if (grouped) {
        for (int32_t s = 0; s < S; ++s) { free(groups[s].val); free(groups[s].cnt); }
        free(groups);
    }
    return 0;
}

/* Exact S at selected (c, k, m) triples, one term per sample. */
int oracle_S_exact_at(int32_t C, const int64_t *offsets, const int32_t *seg, const int32_t *xi,
                      const int32_t *L, const int32_t *eta, const float *lam, const float *cp,
                      const float *cw, int32_t P, const int32_t *cs, const int32_t *ks,
                      const int32_t *ms, int64_t *S_hi, uint64_t *S_lo)
{
    (void)C;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int32_t p = 0; p < P; ++p) {
        int ok = 1;
        int32_t c = cs[p], k = ks[p], m = ms[p], s = seg_of(seg, c);
        int64_t CP = to_fix(cp[c], &ok), CW = to_fix(cw[c], &ok), G = to_fix(lam[m], &ok);
        i128 acc = 0;
        for (int64_t n = offsets[s]; n < offsets[s + 1]; ++n)
            acc += (i128)phi_fix(eta[k], xi[n], L[c], CP, CW, G);
        S_hi[p] = (int64_t)(acc >> 64);
        S_lo[p] = (uint64_t)acc;
        if (!ok) bad = 1;
    }
    return bad ? -1 : 0;
}

/* RN64 of an exact 128-bit fixed-point value, in real units. */
double oracle_fix_to_double(int64_t hi, uint64_t lo)
{
    i128 v = ((i128)hi << 64) | (i128)lo;
    return ldexp((double)v, -FIX_SHIFT);
}

/* out[i] = RN64 of (hi[i], lo[i]) for n values (oracle_fix_to_double over an array). */
void oracle_fix_to_double_n(int64_t n, const int64_t *hi, const uint64_t *lo, double *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_fix_to_double(hi[i], lo[i]);
}

/* J = RN(RN(lam*eps) + RN(RN(S)/N)); lam*eps is exact in double. */
double oracle_J(int64_t hi, uint64_t lo, float lam, float eps, int64_t N)
{
    double s = oracle_fix_to_double(hi, lo);
    double a = (double)lam * (double)eps;
    double b = s / (double)N;
    return a + b;
}

/* W[(e*C + c)*K + k] = min over m of J, mstar = lowest m attaining it. */
void oracle_W(int32_t C, int32_t K, int32_t M, int32_t E, const float *lam, const float *eps,
              const int64_t *N, const int64_t *S_hi, const uint64_t *S_lo, double *W,
              int32_t *mstar)
{
    for (int32_t e = 0; e < E; ++e)
        for (int32_t c = 0; c < C; ++c)
            for (int32_t k = 0; k < K; ++k) {
                double best = INFINITY;
                int32_t bm = 0;
                for (int32_t m = 0; m < M; ++m) {
                    int64_t idx = (int64_t)c * K * M + (int64_t)k * M + m;
                    double j = oracle_J(S_hi[idx], S_lo[idx], lam[m], eps[e * C + c], N[c]);
                    if (j < best) { best = j; bm = m; }
                }
                int64_t o = ((int64_t)e * C + c) * K + k;
                W[o] = best;
                if (mstar) mstar[o] = bm;
            }
}

/* k*[e*C + c] = lowest k <= kmax[c] with the smallest W; Wstar = W there. */
void oracle_argmin(int32_t C, int32_t K, int32_t E, const double *W, const int32_t *kmax,
                   int32_t *kstar, double *Wstar)
{
    for (int32_t e = 0; e < E; ++e)
        for (int32_t c = 0; c < C; ++c) {
            int32_t hi = kmax ? kmax[c] : K - 1;
            if (hi > K - 1) hi = K - 1;
            if (hi < 0) hi = 0;
            const double *w = W + ((int64_t)e * C + c) * K;
            int32_t bk = 0;
            for (int32_t k = 1; k <= hi; ++k)
                if (w[k] < w[bk]) bk = k;
            kstar[e * C + c] = bk;
            Wstar[e * C + c] = w[bk];
        }
}

/* ------------------------------------------------------------- quantile -- */

/* Smallest j in [1, N] with j (c_p + c_w) >= c_p N, in exact integers. */
int64_t oracle_rank(float cp, float cw, int64_t N)
{
    int ok = 1;
    i128 P = to_fix(cp, &ok), Wc = to_fix(cw, &ok);
    if (!ok || N <= 0 || P <= 0 || Wc <= 0) return -1;
    i128 num = P * (i128)N, den = P + Wc;
    i128 j = (num + den - 1) / den;
    if (j < 1) j = 1;
    if (j > N) j = N;
    return (int64_t)j;
}

void oracle_quantile(int32_t C, const int64_t *offsets, const int32_t *seg, const int32_t *xi,
                     const float *cp, const float *cw, int32_t *q_value, int64_t *q_rank)
{
    for (int32_t c = 0; c < C; ++c) {
        int32_t s = seg_of(seg, c);
        int64_t n = offsets[s + 1] - offsets[s];
        int64_t j = oracle_rank(cp[c], cw[c], n);
        q_rank[c] = j;
        if (j < 1) { q_value[c] = -1; continue; }
        int32_t *tmp = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
        memcpy(tmp, xi + offsets[s], sizeof(int32_t) * (size_t)n);
        qsort(tmp, (size_t)n, sizeof(int32_t), cmp_i32);
        q_value[c] = tmp[j - 1];
        free(tmp);
    }
}

/* ----------------------------------------------------------- block step -- */

/* Capacity bound of class c on every group it is routed to, given the other
 * classes' current grid points (the memory-capacity constraint of Sec. 3.4,
 * no prefix caching):
 *   other_g = (1+kappa) * sum_{c' != c} conc[c',g] * eta[k[c']]   (ascending c')
 *   bound_g = (cap[g] - other_g) / ((1+kappa) * conc[c,g])
 * Returns the smallest bound over the groups with conc[c,g] > 0 (+inf if none). */
static double class_bound(int32_t C, int32_t G, int32_t c, const int32_t *eta, const int32_t *kcur,
                          const float *cap, const float *conc, float kappa)
{
    double onek = 1.0 + (double)kappa;
    double bound = INFINITY;
    for (int32_t g = 0; g < G; ++g) {
        double u = (double)conc[c * G + g];
        if (!(u > 0.0)) continue;
        double sum = 0.0;
        for (int32_t c2 = 0; c2 < C; ++c2) {
            if (c2 == c) continue;
            double t = (double)conc[c2 * G + g] * (double)eta[kcur[c2]];
            sum = sum + t;
        }
        double other = onek * sum;
        double num = (double)cap[g] - other;
        double den = onek * u;
        double b = num / den;
        if (b < bound) bound = b;
    }
    return bound;
}

/* One Gauss-Seidel sweep over the classes.  W is the [C*K] table of one radius. */
void oracle_bcd_step(int32_t C, int32_t K, const int32_t *eta, const double *W, int32_t G,
                     const float *cap, const float *conc, float kappa, const int32_t *k_prev,
                     int32_t *k_next, double *W_star, double *usage, uint8_t *feasible)
{
    int32_t *kcur = (int32_t *)malloc(sizeof(int32_t) * (size_t)C);
    memcpy(kcur, k_prev, sizeof(int32_t) * (size_t)C);
    for (int32_t c = 0; c < C; ++c) {
        double bound = class_bound(C, G, c, eta, kcur, cap, conc, kappa);
        int32_t kmax = -1;
        for (int32_t k = 0; k < K; ++k)
            if ((double)eta[k] <= bound) kmax = k;
        feasible[c] = kmax >= 0;
        if (kmax < 0) kmax = 0;
        const double *w = W + (int64_t)c * K;
        int32_t bk = 0;
        for (int32_t k = 1; k <= kmax; ++k)
            if (w[k] < w[bk]) bk = k;
        kcur[c] = bk;
    }
    double onek = 1.0 + (double)kappa;
    for (int32_t g = 0; g < G; ++g) {
        double sum = 0.0;
        for (int32_t c = 0; c < C; ++c) {
            double t = (double)conc[c * G + g] * (double)eta[kcur[c]];
            sum = sum + t;
        }
        usage[g] = onek * sum;
    }
    for (int32_t c = 0; c < C; ++c) {
        k_next[c] = kcur[c];
        W_star[c] = W[(int64_t)c * K + kcur[c]];
    }
    free(kcur);
}

/* Alg. 1 initialisation r0 = L_in + E[xi]: the largest grid point not above
 * the class sample mean (mean compared exactly as sum <= eta * N). */
void oracle_bcd_init(int32_t C, const int64_t *offsets, const int32_t *seg, const int32_t *xi,
                     int32_t K, const int32_t *eta, int32_t *k0)
{
    for (int32_t c = 0; c < C; ++c) {
        int32_t s = seg_of(seg, c);
        int64_t n = offsets[s + 1] - offsets[s], sum = 0;
        for (int64_t i = offsets[s]; i < offsets[s + 1]; ++i) sum += xi[i];
        int32_t best = 0;
        for (int32_t k = 0; k < K; ++k)
            if ((i128)eta[k] * n <= (i128)sum) best = k;
        k0[c] = best;
    }
}

/* ----------------------------------------------- reservation cost, moments -- */

/* Per class: number of samples, their sum, their sum of squares and the
 * largest sample, in exact integers. */
void oracle_moments(int32_t C, const int64_t *offsets, const int32_t *seg, const int32_t *xi,
                    int64_t *count, int64_t *sum, int64_t *sumsq, int32_t *xmax)
{
    for (int32_t c = 0; c < C; ++c) {
        int32_t s = seg_of(seg, c);
        int64_t n = 0, a = 0, b = 0;
        int32_t mx = 0;
        for (int64_t i = offsets[s]; i < offsets[s + 1]; ++i) {
            n += 1;
            a += xi[i];
            b += (int64_t)xi[i] * xi[i];
            if (xi[i] > mx) mx = xi[i];
        }
        count[c] = n;
        sum[c] = a;
        sumsq[c] = b;
        xmax[c] = mx;
    }
}

/* Average stochastic cost of a reservation over the samples of a class
 * (Sec. 3.3, the per-arrival preemption/waste cost of a reservation):
 *   cost[r*C + c]  = RN( RN(S) / N_c ),  S = sum_n Q(eta, x_n) exactly,
 *                    Q(eta, x) = c_p (x - eta)^+ + c_w (eta - x)^+,
 *                    eta = eta_r[r*C + c], any integer;
 *   cover[r*C + c] = #{n : x_n <= eta}   (the empirical level of eta).
 * Every term is an exact multiple of 2^-33 and is summed in 128-bit integers
 * in sample order.  Returns 0, or -1 if a cost is outside the fixed-point range. */
int oracle_reservation_cost(int32_t C, const int64_t *offsets, const int32_t *seg,
                            const int32_t *xi, const float *cp, const float *cw, int32_t R,
                            const int32_t *eta_r, double *cost, int64_t *cover, int64_t *S_hi,
                            uint64_t *S_lo)
{
    int ok = 1;
    for (int32_t c = 0; c < C; ++c) { (void)to_fix(cp[c], &ok); (void)to_fix(cw[c], &ok); }
    if (!ok) return -1;
    int64_t total = (int64_t)R * C;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t rc = 0; rc < total; ++rc) {
        int32_t c = (int32_t)(rc % C);
        int32_t s = seg_of(seg, c);
        int okl = 1;
        i128 CP = to_fix(cp[c], &okl), CW = to_fix(cw[c], &okl);
        i128 eta = eta_r[rc];
        i128 acc = 0;
        int64_t below = 0;
        for (int64_t n = offsets[s]; n < offsets[s + 1]; ++n) {
            i128 x = xi[n];
            i128 q = CP * (x > eta ? x - eta : 0) + CW * (eta > x ? eta - x : 0);
            acc += q;
            if (x <= eta) below += 1;
        }
        int64_t N = offsets[s + 1] - offsets[s];
        double sd = ldexp((double)acc, -FIX_SHIFT);
        cost[rc] = sd / (double)N;
        cover[rc] = below;
        if (S_hi) S_hi[rc] = (int64_t)(acc >> 64);
        if (S_lo) S_lo[rc] = (uint64_t)acc;
    }
    return 0;
}
