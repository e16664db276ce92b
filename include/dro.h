/*
 * dro.h -- C ABI of the MI355X (gfx950) Wasserstein-DRO KV-reservation path.
 *
 * The path evaluates, for every request class c, reservation level eta_k,
 * multiplier lam_m standing in for the Wasserstein dual variable gamma, and
 * historical output-length sample x_n, the per-sample worst-case cost
 *
 *   phi(eta, x, g) = max{ c_w eta - g x,                          candidate at 0
 *                         c_p (x - eta)^+ + c_w (eta - x)^+,       candidate at the sample
 *                         c_p (L - eta) - g (L - x) }              candidate at L_max
 *
 * (paper, Appendix A, Step 4; eta = r - L_in is the buffer of Prop. 4.2),
 * the sums S[c,k,m] = sum_n phi (Appendix A, Step 5), the dual values
 * J = lam_m eps + S / N_c (the Kantorovich dual of Appendix A, Step 3, with gamma on a grid), their
 * minimum over m, the lowest-index argmin over k (the optimal reservation of
 * Prop. 4.2 on the grid), the critical-fractile quantile (Prop. 4.2,
 * eps = 0) and one capacity-constrained reservation update of
 * Block 1 of Alg. 1 under the memory-capacity constraint (Sec. 3.4).
 *
 * Conventions, binding on every entry point:
 *  - Array arguments are DEVICE memory owned by the caller unless the field
 *    name ends in `_h` (HOST memory).  The library never frees or retains a
 *    caller pointer after the call returns; scratch memory belongs to the ctx.
 *  - Every compute call is asynchronous on `stream` (a hipStream_t; NULL is
 *    the null stream): it returns after enqueueing, outputs are valid after
 *    the stream is synchronised.  dro_validate is synchronous.
 *  - Return value 0 = DRO_OK, negative = error.  Nothing is thrown across the
 *    ABI.  On an error found on the host no kernel is launched and no output
 *    is written; dro_last_error(ctx) holds the detail.
 *  - Hot calls check host-visible arguments only.  Device data (sample range,
 *    grid order, coefficient range) is checked by dro_validate; kernels never
 *    read outside the segments given by the offsets, whatever the data.
 *  - A ctx is not thread-safe: use one ctx per host thread / stream.
 *  - Exactness limits (DRO_ELIMIT when exceeded): 0 <= x, eta <= L <= 2^15,
 *    N_c <= 2^26 samples per class, every lam, c_p, c_w in [2^-10, 2^7].
 *    Inside them every candidate of phi is a multiple of 2^-33 below 2^56, so
 *    the library can evaluate S exactly in 128-bit fixed point where the
 *    result is an index (argmin, quantile) or the reported optimum.
 *
 * Layout: tables are row-major, class-major:
 *    S      [C][K][M]      fp64
 *    W      [E][C][K]      fp64     (row e of the radii, class c, grid point k)
 *    m_star [E][C][K]      int32
 *    eps    [E][C]         fp32     radius in tokens (W1 is over output length)
 */
#ifndef DRO_H
#define DRO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct dro_ctx dro_ctx;
typedef void *dro_stream_t; /* a hipStream_t */

enum {
    DRO_OK = 0,
    DRO_EINVAL = -1, /* null pointer, C/K/M/E/S <= 0, bad host offsets, bad segment map */
    DRO_ERANGE = -2, /* device data outside its domain (reported by dro_validate)        */
    DRO_ENOMEM = -3, /* workspace allocation failed                                      */
    DRO_EHIP = -4,   /* HIP runtime error; dro_last_error keeps its text                 */
    DRO_ELIMIT = -5  /* beyond the exactness limits above                                */
};

/* Status bits accumulated on the device by the argmin refine; read and
 * cleared with dro_take_flags. */
enum {
    DRO_FLAG_BAND_FULL = 1u,   /* a screening band held more candidates than the refine keeps */
    DRO_FLAG_BAND_MARGIN = 2u  /* the exact optimum sat too close to the band edge            */
};

/* The reservation sub-problem of one set of classes (paper, Sec. 3.4 and
 * Appendix A, Step 1): samples of the output length per class, the support
 * bound, the reservation grid, the multiplier grid and the two unit costs. */
typedef struct {
    int32_t C;                /* number of request classes                                    */
    int32_t S;                /* number of sample segments; offsets has S+1 entries           */
    const int64_t *offsets;   /* [S+1] ascending CSR bounds into xi, offsets[0] = 0            */
    const int64_t *offsets_h; /* HOST copy of offsets (launch planning); must match            */
    const int32_t *seg;       /* [C] segment of each class, NULL = identity (S = C)            */
    const int32_t *seg_h;     /* HOST copy of seg, NULL iff seg is NULL                        */
    const int32_t *xi;        /* samples of the output length, 0 <= x <= L[c]                  */
    const int32_t *L;         /* [C] support bound L_max of each class (Xi = [0, L])           */
    int32_t K;
    const int32_t *eta;       /* [K] strictly ascending buffer levels eta = r - L_in, in [0,L] */
    int32_t M;
    const float *lam;         /* [M] strictly ascending multipliers > 0 (gamma on a grid)       */
    const float *c_p;         /* [C] preemption cost per token (Sec. 3.3)                       */
    const float *c_w;         /* [C] waste cost per reserved, unused token (Sec. 3.3)           */
} dro_problem;

/* Serving groups for the capacity constraint (the memory-capacity constraint of Sec. 3.4, no prefix caching). */
typedef struct {
    int32_t G;
    const float *cap;         /* [G] KV capacity of each group, tokens (M_k)                    */
    const float *conc;        /* [C][G] expected concurrent class-c requests on group g (>= 0,   */
                              /*        0 = not routed): u_{i,k} pi_{i,k} / z_k                  */
    float kappa;              /* concurrency safety factor (Sec. 5.1 uses 0.2)                  */
} dro_groups;

typedef struct {
    int32_t *k_next;          /* [C] updated grid index of each class                          */
    double *W_star;           /* [C] exact dual value at k_next                                 */
    int32_t *q_value;         /* [C] critical-fractile quantile of each class                   */
    double *usage;            /* [G] (1+kappa) sum_c conc[c,g] eta[k_next[c]]                   */
    uint8_t *feasible;        /* [C] 1 if some grid point met every capacity bound              */
} dro_step_out;

const char *dro_strerror(int code);

/* Create a context on HIP device `hip_device` (made current by every call). */
int dro_create(int hip_device, dro_ctx **out);
void dro_destroy(dro_ctx *ctx);
const char *dro_last_error(const dro_ctx *ctx);

/* Synchronous check of the device data of `p` (and of eps[E*C] when E > 0):
 * sample range, segment map, grid order and range, coefficient range, host
 * offsets equal to the device offsets.  Returns DRO_ERANGE or DRO_ELIMIT
 * with a message naming the first violation found. */
int dro_validate(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                 dro_stream_t stream);

/* Read and clear the DRO_FLAG_* bits raised since the last call (synchronous). */
int dro_take_flags(dro_ctx *ctx, uint32_t *flags_out);

/* Dense evaluation (Appendix A, Steps 4-5) and the minimum over the
 * multiplier grid (Kantorovich dual, Appendix A, Step 3):
 *   S[c,k,m]  = sum over the samples of class c of phi(eta_k, x, lam_m)
 *               every (c,k,m,n) term in fp32, runs of at most 64 samples
 *               folded into fp64 in a fixed order (deterministic)
 *   W[e,c,k]  = min over m of  RN(RN(lam_m eps[e,c]) + RN(S[c,k,m] / N_c))
 *   m_star    = the lowest m attaining it.
 * S may be NULL (kept in the ctx workspace); m_star may be NULL.
 * W is accurate to about 1e-7 relative; use dro_argmin_reservation for the
 * exact optimum. */
int dro_cost_eval(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps, double *W,
                  int32_t *m_star, double *S, dro_stream_t stream);

/* Optimal grid reservation per (e, c) (Prop. 4.2 on the grid):
 *   k_star[e,c]    = lowest k <= k_max[c] minimising min_m J   (k_max NULL = K-1)
 *   W_star[e,c]    = exact J at the optimum: J = RN(RN(lam eps) + RN(RN(S)/N)) with S
 *                    the exact sum of phi (128-bit fixed point), round-to-nearest-even
 *   m_at_star[e,c] = lowest m attaining it (may be NULL).
 * `S` is the table written by dro_cost_eval for the same problem; it is used to
 * screen candidates, which are then evaluated exactly.  Ties go to the lowest k,
 * then the lowest m. */
int dro_argmin_reservation(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                           const double *S, const int32_t *k_max, int32_t *k_star, double *W_star,
                           int32_t *m_at_star, dro_stream_t stream);

/* Critical-fractile quantile per class (Prop. 4.2 at eps = 0,
 * generalized inverse of the empirical CDF):
 *   q_rank[c]  = j = ceil(c_p N_c / (c_p + c_w)), computed exactly, in [1, N_c]
 *   q_value[c] = the j-th smallest sample of class c.
 * Uses C, S, offsets, seg, xi, L, c_p, c_w of `p`. */
int class_quantile(dro_ctx *ctx, const dro_problem *p, int32_t *q_value, int64_t *q_rank,
                   dro_stream_t stream);

/* Exact table by value grouping and prefix sums.  For 0 <= x, eta <= L the three
 * candidates of Step 4 reduce to the larger of two lines in x, so with the
 * per-segment counts and sums of the sample values every S[c,k,m] is a closed
 * form in 128-bit integers: O(N + L) per segment plus O(1) per (c,k,m), instead
 * of O(N) per (c,k,m).  This is the production alternative to the dense
 * evaluation when only the results are needed (it does not evaluate every
 * per-sample term, so it is not the dense throughput measurement):
 *   W[e,c,k], m_star[e,c,k] = exact-spec values (the expression of
 *                             dro_argmin_reservation for every k), lowest m
 *   k_star, W_star, m_at_star [E*C] = lowest-index optimum with k <= k_max[c]
 *                             (k_star NULL: the argmin is skipped; m_at_star may be NULL).
 * Uses C, S, offsets, seg, xi, L, eta, lam, c_p, c_w of `p`; k_max may be NULL. */
int dro_exact_table(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                    const int32_t *k_max, double *W, int32_t *m_star, int32_t *k_star,
                    double *W_star, int32_t *m_at_star, dro_stream_t stream);

/* Continuous-multiplier dual (Kantorovich dual of Appendix A, Step 3, with
 * gamma >= 0 continuous; equal to the LP of Step 5 by strong duality, Step 2):
 *   W[e,c,k]     = min over gamma >= 0 of gamma eps[e,c] + S(gamma) / N_c
 *   gamma[e,c,k] = the smallest minimising gamma (in [0, max(c_p, c_w)])
 * J is convex and piecewise linear in gamma; its right derivative follows from
 * the per-segment value counts and sums, and a bisection finds the smallest
 * minimiser; values are fp64 (relative error ~1e-12), not the exact-spec
 * expression.  This removes the multiplier grid: W here is <= the grid W of
 * dro_cost_eval, with equality when the grid holds the minimiser. */
int dro_continuous_dual(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                        double *W, double *gamma, dro_stream_t stream);

/* Per-class sample moments, exact (the inputs of the mean-based reservation of
 * Alg. 1's initial state and of the mean and mean-plus-spread baselines of
 * Sec. 5.1 and Sec. 5.4):
 *   count[c] = N_c,  sum[c] = sum of x,  sumsq[c] = sum of x^2,
 *   xmax[c]  = the largest sample of class c.
 * All outputs are device arrays of length C.  Uses C, S, offsets, seg, xi, L of
 * `p` (the value histogram assumes validated samples, 0 <= x <= L <= 2^15). */
int class_moments(dro_ctx *ctx, const dro_problem *p, int64_t *count, int64_t *sum,
                  int64_t *sumsq, int32_t *xmax, dro_stream_t stream);

/* Average stochastic cost of given reservations over each class's samples
 * (the per-arrival preemption/waste cost of Sec. 3.3 with eta = r - L_in, by
 * which Sec. 5.2 and Table 2 compare reservation policies):
 *   cost[r*C + c]  = RN( RN(S) / N_c ),  S = sum_n Q(eta, x_n) exactly,
 *                    Q(eta, x) = c_p (x - eta)^+ + c_w (eta - x)^+,
 *   cover[r*C + c] = #{n : x_n <= eta}, the empirical level of eta,
 * for eta = eta_r[r*C + c], r = 0..R-1.  eta_r is a device int32 array of
 * R*C reservations (any integer: below 0 every sample is preempted, above the
 * largest sample every one is waste); cost (double) and cover (int64) are
 * device arrays of R*C.  Exact: the sum follows from the per-segment value
 * counts and sums in 128-bit integers.  R >= 1 and all pointers non-NULL, else
 * DRO_EINVAL.  Uses C, S, offsets, seg, xi, L, c_p, c_w of `p`. */
int dro_reservation_cost(dro_ctx *ctx, const dro_problem *p, int32_t R, const int32_t *eta_r,
                         double *cost, int64_t *cover, dro_stream_t stream);

/* Initial state of Alg. 1: r0 = L_in + E[xi], i.e. k0[c] = the largest k with
 * eta[k] <= mean of the class samples (compared exactly). */
int bcd_init_state(dro_ctx *ctx, const dro_problem *p, int32_t *k0, dro_stream_t stream);

/* One reservation update of Block 1 of Alg. 1 under the memory-capacity
 * constraint (Sec. 3.4):
 * class_quantile, dro_cost_eval with one radius row eps[C], then a
 * Gauss-Seidel sweep over c = 0..C-1 in order.  For class c, with the other
 * classes at their current grid points and for every group g with
 * conc[c,g] > 0 (fp64, no contraction, sums in ascending class order):
 *   other_g = (1+kappa) * sum_{c' != c} conc[c',g] * eta[k[c']]
 *   bound_g = (cap[g] - other_g) / ((1+kappa) * conc[c,g])
 *   kmax_c  = the largest k with eta[k] <= min_g bound_g
 *             (none: kmax_c = 0 and feasible[c] = 0)
 *   k[c]    = lowest argmin over k <= kmax_c of the exact W[c,k].
 * k_prev[C] is the state entering the sweep. */
int bcd_block_step(dro_ctx *ctx, const dro_problem *p, const float *eps, const dro_groups *g,
                   const int32_t *k_prev, dro_step_out *out, dro_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DRO_H */
