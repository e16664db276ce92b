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
 * Further entry points: the same table exactly from value counts, the
 * dual over continuous gamma, per-class moments and the cost of given
 * reservations (the policy comparison of Sec. 5), and the rest of Alg. 1
 * (routing LP, prefix caching, configuration search; last section).
 *
 * Conventions, binding on every entry point:
 *  - Array arguments are DEVICE memory owned by the caller unless the field
 *    name ends in `_h` (HOST memory).  The library never frees or retains a
 *    caller pointer after the call returns; scratch memory belongs to the ctx.
 *  - Every compute call is asynchronous on `stream` (a hipStream_t; NULL is
 *    the null stream): it returns after enqueueing, outputs are valid after
 *    the stream is synchronised.  dro_validate and dro_bcd_solve (whose loop
 *    reads its decisions on the host) are synchronous.
 *  - Return value 0 = DRO_OK, negative = error.  Nothing is thrown across the
 *    ABI.  On an error found on the host no kernel is launched and no output
 *    is written; dro_last_error(ctx) holds the detail.
 *  - Hot calls check host-visible arguments only.  Device data (sample range,
 *    grid order, coefficient range) is checked by dro_validate; kernels never
 *    read outside the segments given by the offsets, whatever the data.
 *  - A ctx is not thread-safe: use one ctx per host thread / stream.
 *  - HIP graphs: once a call has run with the same problem on the same stream
 *    (sizing the workspace and staging the offsets), class_quantile,
 *    dro_cost_eval and dro_argmin_reservation enqueue kernels only, with no
 *    allocation, host copy or memset, so a stream capture of them replays
 *    correctly.
 *  - Exactness limits (DRO_ELIMIT when exceeded): 0 <= x, eta <= L <= 2^15,
 *    N_c <= 2^26 samples per class, every lam, c_p, c_w in [2^-10, 2^7];
 *    K <= 2^15 + 1 grid points, M <= 65536 multipliers, K * M < 2^31 pairs,
 *    E * C < 2^31 radius rows, and (dense evaluation) fewer than 2^31 - 1
 *    tiles of 8192 (k, m) pairs over all classes.
 *    Inside them every candidate of phi is a multiple of 2^-33 below 2^56, so
 *    the library evaluates every S exactly in 128-bit fixed point and rounds
 *    it to double once.
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

/* Dense evaluation (Appendix A, Steps 4-5) and the minimum over the
 * multiplier grid (Kantorovich dual, Appendix A, Step 3):
 *   S[c,k,m]  = sum over the samples of class c of phi(eta_k, x, lam_m), exactly:
 *               every (c,k,m,n) term's per-sample part |x - t| (t the integer
 *               floor or ceiling of the crossing point of phi's two lines) is
 *               summed in integers on the GPU, and the rest of each term follows
 *               from N, the sample sum and one value count per (c,k,m); S is the
 *               correctly rounded double of the exact sum (deterministic)
 *   W[e,c,k]  = min over m of  RN(RN(lam_m eps[e,c]) + RN(S[c,k,m] / N_c))
 *   m_star    = the lowest m attaining it.
 * S may be NULL (kept in the ctx workspace); m_star may be NULL.  Inside the
 * exactness limits S, W and m_star are exact for every cost ratio: the same
 * values as the exact-spec expression of dro_argmin_reservation. */
int dro_cost_eval(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps, double *W,
                  int32_t *m_star, double *S, dro_stream_t stream);

/* Bytes of the device array that dro_cost_eval_noalloc takes its scratch from
 * (one array per device, held until the process ends). */
#define DRO_NOALLOC_SCRATCH_BYTES (32u << 20)

/* dro_cost_eval for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, results and errors as dro_cost_eval, except that S is
 * required (the dense sums accumulate in it) and the scratch (the staged
 * offsets and segment map, the value histogram, the prefix counts and sums,
 * the dense kernel's work counters, one per tile) comes from a static device array of DRO_NOALLOC_SCRATCH_BYTES instead of
 * the ctx workspace, so the call allocates nothing.  The scratch grows with
 * the number of sample segments, about 0.5 MB each: a problem that needs
 * more than the array (beyond about 60 segments) gets DRO_ELIMIT before any
 * work is enqueued.  Every call on one device shares that device's array and
 * leaves its contents behind; two calls that overlap on one device (from
 * different streams or host threads) race. */
int dro_cost_eval_noalloc(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                          double *W, int32_t *m_star, double *S, dro_stream_t stream);

/* Optimal grid reservation per (e, c) (Prop. 4.2 on the grid):
 *   k_star[e,c]    = lowest k <= k_max[c] minimising W[e,c,k] = min_m J   (k_max NULL = K-1)
 *   W_star[e,c]    = J at the optimum: J = RN(RN(lam eps) + RN(S/N)), round-to-nearest-even
 *   m_at_star[e,c] = lowest m attaining it (may be NULL).
 * `S` is the table written by dro_cost_eval for the same problem: the
 * correctly rounded double of the exact sum, so every J is the exact-spec
 * value and the optimum is exact.  Ties go to the lowest k, then the lowest m. */
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

/* The moment-based and block-aligned baseline reservations that the policy
 * comparison prices against DRO (Sec. 5.1: the mean and P95 with block
 * alignment; Sec. 5.4: mean plus k standard deviations), exactly in integers,
 * from the per-class count n, sum s and sum of squares ss of class_moments:
 *   mean_r[c]       = ceil(s / n), the least integer >= the mean
 *   lp_r[i*C + c]   = min(L[c], the least integer >= mean + k_i sigma), sigma
 *                     the population standard deviation; equivalently
 *                     ceil((s + ceil(sqrt(k_i^2 (n ss - s^2)))) / n)
 *   block_r[c]      = q[c] rounded up to a multiple of `block` tokens
 * for i = 0..nk-1 with k_i = k_sigma_h[i] (HOST array, integers in [0, 64],
 * nk <= 8).  count, sum, sumsq (int64), L, q (int32) and the outputs (int32)
 * are device arrays of length C (lp_r: nk*C); q and block_r are NULL together
 * (block >= 1 when given), lp_r and k_sigma_h may be NULL when nk = 0.
 * Violations give DRO_EINVAL before any work is enqueued.  The square root is
 * a double estimate corrected with exact 128-bit products. */
int dro_baseline_reservations(dro_ctx *ctx, int32_t C, const int64_t *count, const int64_t *sum,
                              const int64_t *sumsq, const int32_t *L, int32_t nk,
                              const int32_t *k_sigma_h, const int32_t *q, int32_t block,
                              int32_t *mean_r, int32_t *lp_r, int32_t *block_r,
                              dro_stream_t stream);

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

/* ------------------------------------------------------------------------
 * The rest of Alg. 1 (Sec. 4.3): the routing LP of Block 1 (LP1), prefix
 * caching (Block 2) and the configuration search (Block 3), over the serving
 * model of Sec. 3.1-3.4.  For class c and configuration g (z_g serving groups
 * of tau_g x pp_g GPUs each):
 *   T[c,g]    = pp_g alpha Lin_c / Cc_g + NL tau_g t_ar + beta E[xi_c] / Bc_g
 *               (service time, Sec. 3.1, with E[xi_c] the class sample mean)
 *   ET2[c,g]  = its second moment over the class samples
 *   conc[c,g] = lam_c T_cg pi_cg / z_g   (concurrent requests, Little's law)
 *   mem[g]    = (1 + kappa) (sum_c lam_c T_cg pi_cg (Lin_c + eta_c - delta_cg Lpre_c)) / z_g
 *               + sum_c delta_cg Lpre_c   (KV tokens in use, the memory-capacity
 *               constraint of Sec. 3.4 with r~ = r - delta L_pre, r = Lin + eta)
 *   Wq[g]     = u (1 + Cs2) / (2 (1 - u)) Tbar, u = mem_g / Mcap_g: the
 *               Pollaczek-Khinchin wait of Sec. 3.4 at the memory utilisation,
 *               Tbar and Cs2 the mean and squared coefficient of variation of
 *               the routed service times (Wq = 0 without traffic)
 *   objective = sum_c lam_c (a_c W_c + sum_g pi_cg c_gpu tau_g pp_g T_cg + c_slo s_c
 *               + (1 - a_c) c_rej), a_c = sum_g pi_cg,
 *               s_c = max(0, sum_g pi_cg (Wq_g + T_cg) - a_c D_c)   (Prop. 4.1)
 *   feasible  : sum_g z_g tau_g pp_g <= J; pi_cg > 0 only where z_g > 0;
 *               mem_g <= u_max Mcap_g (1 + 1e-9) (u_max < 1 keeps the wait
 *               finite; the slack keeps a routing that an LP left exactly at the
 *               bound feasible).
 * All double expressions are evaluated in a fixed order without contraction.
 * Limits: 1 <= G <= 32, C * G <= 8192, 1 <= J <= 4096 and at most 2^32
 * configurations in the search space, else DRO_ELIMIT.
 * ---------------------------------------------------------------------- */
typedef struct {
    int32_t G;                 /* candidate configurations */
    const int32_t *tau, *pp;   /* device [G] tensor / pipeline degree (>= 1) */
    const int32_t *tau_h, *pp_h; /* host copies of tau and pp */
    const float *Mcap;         /* device [G] KV capacity of one group, tokens */
    const float *Cc, *Bc;      /* device [G] prefill and decode rates, tokens/s */
    const float *lam;          /* device [C] arrival rate, requests/s */
    const int32_t *Lin, *Lpre; /* device [C] input length and cacheable prefix, tokens */
    const float *D;            /* device [C] latency target, s */
    float alpha, beta, t_ar;   /* prefill and decode constants, all-reduce latency (s) */
    int32_t NL;                /* layers */
    float c_gpu, c_slo, c_rej; /* cost per GPU-second, per second late, per rejection */
    float kappa, u_max;        /* memory-headroom factor; utilisation bound in (0, 1) */
    int32_t J;                 /* GPU budget */
} dro_service;

/* T and ET2 (device double [C*G], row c*G + g) from the exact class moments.
 * Uses C, S, offsets, seg, xi, L of `p`. */
int bcd_service_times(dro_ctx *ctx, const dro_problem *p, const dro_service *svc, double *T,
                      double *ET2, dro_stream_t stream);

/* Per configuration at a given state (all device arrays; pi, conc [C*G];
 * z, Wq, cap, mem [G]; eta_c [C] = each class's reservation beyond its input;
 * delta [C*G] 0/1): Wq, mem (may be NULL), conc, and
 *   cap[g] = u_max Mcap_g - sum_c delta_cg Lpre_c
 *            - (1 + kappa) (sum_c lam_c T_cg pi_cg (Lin_c - delta_cg Lpre_c)) / z_g,
 * the memory left for the reservations (+inf where z_g = 0). */
int bcd_queue_state(dro_ctx *ctx, int32_t C, const dro_service *svc, const double *T,
                    const double *ET2, const double *pi, const int32_t *z, const int32_t *eta_c,
                    const uint8_t *delta, double *Wq, double *cap, double *conc, double *mem,
                    dro_stream_t stream);

/* LP1 of Block 1: the routing pi >= 0 (device [C*G]) minimising the objective
 * with the reservations, z and delta fixed and the wait Wq (device [G]) frozen
 * at the incoming state, subject to sum_g pi_cg <= 1, the SLO slack rows and
 * mem_g <= u_max Mcap_g.  Wc [C] holds each class's worst-case cost at its
 * reservation.  Dense simplex in one workgroup (fp64, rows scaled by their
 * largest coefficient): the most negative reduced cost enters, and after 20
 * degenerate pivots in a row Bland's rule takes over until the objective
 * moves, so the method cannot cycle.  lp_objective (device double [1]) is
 * the objective at the solution with s_c at its optimum; info (device int32
 * [2]) = {pivots, status}: 0 optimal, 1 pivot limit, 2 infeasible at pi = 0
 * (prefixes alone exceed a capacity), 3 unbounded. */
int bcd_routing_lp(dro_ctx *ctx, int32_t C, const dro_service *svc, const double *Wc,
                   const double *T, const double *Wq, const int32_t *z, const int32_t *eta_c,
                   const uint8_t *delta, double *pi, double *lp_objective, int32_t *info,
                   dro_stream_t stream);

/* LP2 of Block 1 on the grid: one Gauss-Seidel sweep over c = 0..C-1 of the
 * exact table W (device double [C*K]): with the other classes at their
 * current grid points, bound_g = (cap_g - (1+kappa) sum_{c' != c} conc_c'g
 * eta[k_c']) / ((1+kappa) conc_cg) over the g with conc_cg > 0, kmax = the
 * largest k with eta[k] <= min_g bound_g + 1e-6 (none: kmax = 0,
 * feasible[c] = 0),
 * k_out[c] = the lowest argmin of W[c, 0..kmax].  feasible may be NULL. */
int bcd_reservation_sweep(dro_ctx *ctx, int32_t C, int32_t K, const double *W,
                          const int32_t *eta, int32_t G, const double *conc, const double *cap,
                          float kappa, const int32_t *k_in, int32_t *k_out, uint8_t *feasible,
                          dro_stream_t stream);

/* Block 2: delta[c*G + g] = 1[conc_cg > 1] (device arrays). */
int bcd_prefix_cache(dro_ctx *ctx, int32_t C, int32_t G, const double *conc, uint8_t *delta,
                     dro_stream_t stream);

/* Block 3: every z in Z = {z >= 0 : sum_g z_g tau_g pp_g <= J}, one thread
 * per z in lexicographic order of (z_0, .., z_{G-1}), evaluated with pi, the
 * reservations and delta fixed; the first minimiser of the objective over the
 * feasible z replaces z (device int32 [G], in/out) unless the incoming z
 * attains the minimum (no feasible z: z is kept).  best_objective (double),
 * best_rank and n_feasible (int64) are device scalars (rank -1: none). */
int bcd_config_search(dro_ctx *ctx, int32_t C, const dro_service *svc, const double *Wc,
                      const double *T, const double *ET2, const double *pi,
                      const int32_t *eta_c, const uint8_t *delta, int32_t *z,
                      double *best_objective, int64_t *best_rank, int64_t *n_feasible,
                      dro_stream_t stream);

/* Alg. 1 with the reservation on the grid.  Start: z (device int32 [G], in),
 * delta = 0, pi = 0, reservations at the largest grid point not above the
 * class mean (Alg. 1 init); the worst-case table W[c,k] of radius row eps[C]
 * is computed once, exactly (as dro_exact_table).  Block 1 takes the wait Wq
 * at the state entering it and alternates bcd_routing_lp (with that Wq) and
 * bcd_reservation_sweep until the reservations repeat and max |pi change|
 * <= 1e-9, at most max_inner times; Block 2 sets delta; Block 3 runs bcd_config_search; the
 * loop ends when z and delta repeat, after at most max_outer iterations.
 * Outputs (device): z [G], k [C], pi [C*G], delta [C*G], objective [1] (at
 * the final state).  info (host int32 [4]) = {outer iterations, Block 1
 * rounds, simplex pivots, status bits: 1 pivot limit, 2 infeasible LP start,
 * 4 unbounded LP, 8 a class without a feasible reservation, 16 Block 1 hit
 * max_inner, 32 the loop hit max_outer}.  Synchronises the stream once per
 * Block 1 round (the loop's decisions are read on the host).  Uses every
 * field of `p`. */
int dro_bcd_solve(dro_ctx *ctx, const dro_problem *p, const float *eps, const dro_service *svc,
                  int32_t max_outer, int32_t max_inner, int32_t *z, int32_t *k, double *pi,
                  uint8_t *delta, double *objective, int32_t *info, dro_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DRO_H */
