// The rest of Alg. 1 around the reservation update: the routing LP (LP1 of
// Block 1), prefix caching (Block 2) and the configuration search (Block 3),
// over the serving model of Sec. 3.1-3.4.
//
// Compiled with -ffp-contract=off: every double expression is evaluated in the
// order written, one rounding per operation, so that the decisions taken on
// its values (capacity bounds, the caching threshold, the configuration
// objective) are reproducible bit for bit.
//
// Model (per class c and configuration g; z_g groups of configuration g):
//   T[c,g]    = pp_g alpha Lin_c / Cc_g + NL tau_g t_ar + beta E[xi_c] / Bc_g
//   conc[c,g] = lam_c T_cg pi_cg / z_g                      (Little's law)
//   mem[g]    = (1 + kappa) (sum_c lam_c T_cg pi_cg (Lin_c + eta_c - delta_cg Lpre_c)) / z_g
//               + sum_c delta_cg Lpre_c                      (KV tokens in use)
//   Wq[g]     = u (1 + Cs2) / (2 (1 - u)) Tbar with u = mem_g / Mcap_g
//               (Pollaczek-Khinchin at the memory utilisation)
//   objective = sum_c lam_c (a_c W_c + sum_g pi_cg c_gpu tau_g pp_g T_cg + c_slo s_c
//               + (1 - a_c) c_rej),  s_c = max(0, sum_g pi_cg (Wq_g + T_cg) - a_c D_c)
//   feasible  : sum_g z_g tau_g pp_g <= J, pi_cg > 0 only where z_g > 0,
//               mem_g <= u_max Mcap_g (1 + 1e-9): the slack makes a routing that
//               the LP leaves exactly at its memory bound count as feasible.
#include <cmath>

#include "dro_internal.h"

namespace dro {

namespace {

constexpr int kSvcThreads = 256;
constexpr double kMemSlack = 1.0 + 1e-9;  // relative slack of a configuration's memory check
constexpr double kEtaSlack = 1e-6;        // tokens of slack of the sweep's reservation bound
constexpr int kLpDegenerateRun = 20;      // degenerate pivots before the simplex turns to Bland's rule

__device__ __forceinline__ double block_min_d(double v, double *red)
{
    const int t = threadIdx.x;
    red[t] = v;
    __syncthreads();
    for (int w = blockDim.x / 2; w > 0; w >>= 1) {
        if (t < w && red[t + w] < red[t]) red[t] = red[t + w];
        __syncthreads();
    }
    const double r = red[0];
    __syncthreads();
    return r;
}

// lowest index among the threads' candidates (INT_MAX = none)
__device__ __forceinline__ int block_min_i(int v, int *red)
{
    const int t = threadIdx.x;
    red[t] = v;
    __syncthreads();
    for (int w = blockDim.x / 2; w > 0; w >>= 1) {
        if (t < w && red[t + w] < red[t]) red[t] = red[t + w];
        __syncthreads();
    }
    const int r = red[0];
    __syncthreads();
    return r;
}

// Lexicographic minimum of (key, idx) over the block (smallest key, then the
// smallest idx), carrying aux along: shuffles inside each wave, then one pass
// over the per-wave results in LDS.
struct KeyIdx {
    double key;
    int idx, aux;
};

__device__ __forceinline__ KeyIdx block_min_key(double k, int i, int a, double *sk, int *si,
                                                int *sa)
{
    for (int off = 32; off > 0; off >>= 1) {
        const double k2 = __shfl_xor(k, off);
        const int i2 = __shfl_xor(i, off), a2 = __shfl_xor(a, off);
        if (k2 < k || (k2 == k && i2 < i)) {
            k = k2;
            i = i2;
            a = a2;
        }
    }
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = (blockDim.x + 63) >> 6;
    if (lane == 0) {
        sk[wid] = k;
        si[wid] = i;
        sa[wid] = a;
    }
    __syncthreads();
    KeyIdx r{sk[0], si[0], sa[0]};
    for (int q = 1; q < nw; ++q)
        if (sk[q] < r.key || (sk[q] == r.key && si[q] < r.idx)) r = KeyIdx{sk[q], si[q], sa[q]};
    __syncthreads();
    return r;
}

}  // namespace

// ------------------------------------------------------------ service times --
__global__ void service_times_kernel(SvcArgs s, const int64_t *count, const int64_t *sum,
                                     const int64_t *sumsq, double *T, double *ET2)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= s.C * s.G) return;
    const int c = i / s.G, g = i % s.G;
    const double n = (double)count[c];
    const double mean = (double)sum[c] / n;
    const double ex2 = (double)sumsq[c] / n;
    double A = (double)s.pp[g] * s.alpha * (double)s.Lin[c] / (double)s.Cc[g];
    A = A + s.NL * (double)s.tau[g] * s.t_ar;
    const double B = s.beta / (double)s.Bc[g];
    T[i] = A + B * mean;
    ET2[i] = A * A + 2.0 * A * B * mean + B * B * ex2;
}

// ---------------------------------------------------------------- state -----
// Per configuration g (one thread each): the waiting time at the current
// state, the memory left for the reservations (cap) and conc[c, g].
__global__ void state_kernel(SvcArgs s, const double *T, const double *ET2, const double *pi,
                             const int32_t *z, const int32_t *eta_c, const uint8_t *delta,
                             double *Wq, double *cap, double *conc, double *mem_out)
{
    const int g = blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= s.G) return;
    const int C = s.C, G = s.G;
    if (z[g] <= 0) {
        Wq[g] = 0.0;
        cap[g] = INFINITY;
        if (mem_out) mem_out[g] = 0.0;
        for (int c = 0; c < C; ++c) conc[c * G + g] = 0.0;
        return;
    }
    const double zg = (double)z[g];
    double used = 0.0, fixed = 0.0, pre = 0.0, load = 0.0, X = 0.0, m2 = 0.0;
    for (int c = 0; c < C; ++c) {
        const int i = c * G + g;
        const int dl = delta[i] ? s.Lpre[c] : 0;
        const double lTp = (double)s.lam[c] * T[i] * pi[i];
        used = used + lTp * (double)(s.Lin[c] + eta_c[c] - dl);
        fixed = fixed + lTp * (double)(s.Lin[c] - dl);
        pre = pre + (double)dl;
        conc[i] = lTp / zg;
        const double wgt = (double)s.lam[c] * pi[i];
        load = load + wgt * T[i];
        X = X + wgt;
        m2 = m2 + wgt * ET2[i];
    }
    const double kap = 1.0 + s.kappa;
    const double mem = kap * (used / zg) + pre;
    double w = 0.0;
    if (X > 0.0) {
        const double u = mem / (double)s.Mcap[g];
        const double tb = load / X;
        const double cs2 = (m2 / X) / (tb * tb) - 1.0;
        w = u < 1.0 ? u * (1.0 + cs2) / (2.0 * (1.0 - u)) * tb : INFINITY;
    }
    Wq[g] = w;
    cap[g] = s.u_max * (double)s.Mcap[g] - pre - kap * (fixed / zg);
    if (mem_out) mem_out[g] = mem;
}

// Wc[c] = W[c, k[c]] and eta_c[c] = eta[k[c]]
__global__ void gather_kernel(const double *W, const int32_t *eta, const int32_t *k, int C, int K,
                              double *Wc, int32_t *eta_c)
{
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c < C) {
        const int kc = min(max(k[c], 0), K - 1);
        Wc[c] = W[(long long)c * K + kc];
        eta_c[c] = eta[kc];
    }
}

// Block 2: delta = 1[conc > 1]
__global__ void cache_kernel(const double *conc, int n, uint8_t *delta)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) delta[i] = conc[i] > 1.0 ? 1 : 0;
}

__global__ void zero_u8_kernel(uint8_t *p, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

// ------------------------------------------------------------------- LP1 ----
// min c^T x over x >= 0 with A x <= b, b >= 0, by the simplex method on a
// dense tableau.  The entering column has the most negative reduced cost;
// after 20 degenerate pivots in a row the rule becomes Bland's (smallest
// entering index) until a pivot moves the objective, so the method cannot
// cycle.  Ties of the ratio test go to the smallest basic index.  Variables: pi[c,g]
// at c*G + g (fixed at 0 where z_g = 0), then s_c.  Rows: sum_g pi_cg <= 1;
// sum_g pi_cg (Wq_g + T_cg - D_c) - s_c <= 0; memory of every g with z_g > 0
// (empty rows otherwise).  Each row is scaled by its largest coefficient, the
// objective by its largest cost.  One block; the tableau lives in `tab`
// ((m + 1) x (n + m + 1) doubles), the basis in `basis` (m ints).
__global__ __launch_bounds__(kSvcThreads) void lp1_kernel(
    SvcArgs s, const double *Wc, const double *T, const double *Wq, const int32_t *z,
    const int32_t *eta_c, const uint8_t *delta, double *tab_g, int32_t *basis, double *col_g,
    int in_lds, int max_pivots, double *pi_out, double *obj_out, int32_t *info)
{
    extern __shared__ double lds_tab[];  // (m + 1) * w + (m + 1) doubles when in_lds
    __shared__ double red_d[kSvcThreads];
    __shared__ int red_i[kSvcThreads];
    __shared__ double wk_d[kSvcThreads / 64];
    __shared__ int wk_i[kSvcThreads / 64], wk_a[kSvcThreads / 64];
    __shared__ double sh_scale;
    const int t = threadIdx.x, nt = blockDim.x;
    const int C = s.C, G = s.G;
    const int nv = C * G + C, m = 2 * C + G, w = nv + m + 1;
    const double kap = 1.0 + s.kappa;
    double *tab = in_lds ? lds_tab : tab_g;
    double *col = in_lds ? lds_tab + (long long)(m + 1) * w : col_g;

    // build: constraint rows, slack identity, right-hand sides
    for (long long e = t; e < (long long)(m + 1) * w; e += nt) tab[e] = 0.0;
    __syncthreads();
    bool bad = false;
    for (int r = t; r < m; r += nt) {
        double *row = tab + (long long)r * w;
        double rhs;
        if (r < C) {
            const int c = r;
            for (int g = 0; g < G; ++g) row[c * G + g] = z[g] > 0 ? 1.0 : 0.0;
            rhs = 1.0;
        } else if (r < 2 * C) {
            const int c = r - C;
            for (int g = 0; g < G; ++g)
                if (z[g] > 0) row[c * G + g] = Wq[g] + T[c * G + g] - (double)s.D[c];
            row[C * G + c] = -1.0;
            rhs = 0.0;
        } else {
            const int g = r - 2 * C;
            double pre = 0.0;
            rhs = 0.0;
            if (z[g] > 0) {
                for (int c = 0; c < C; ++c) {
                    const int dl = delta[c * G + g] ? s.Lpre[c] : 0;
                    const double rt = (double)(s.Lin[c] + eta_c[c] - dl);
                    row[c * G + g] = kap * ((double)s.lam[c] * T[c * G + g] / (double)z[g]) * rt;
                    pre += (double)dl;
                }
                rhs = s.u_max * (double)s.Mcap[g] - pre;
            }
        }
        if (rhs < 0.0) bad = true;
        double mx = 0.0;
        for (int j = 0; j < nv; ++j) mx = fmax(mx, fabs(row[j]));
        const double sc = mx > 0.0 ? 1.0 / mx : 1.0;
        for (int j = 0; j < nv; ++j) row[j] *= sc;
        row[nv + r] = 1.0;
        row[w - 1] = rhs * sc;
        basis[r] = nv + r;
    }
    // objective row: reduced costs (the slack basis has zero cost)
    double lmx = 0.0;
    for (int j = t; j < nv; j += nt) {
        double cj;
        if (j < C * G) {
            const int c = j / G, g = j % G;
            cj = z[g] > 0 ? (double)s.lam[c] * (Wc[c] + s.c_gpu * (double)(s.tau[g] * s.pp[g]) *
                                                         T[j] - s.c_rej)
                          : 0.0;
        } else {
            cj = (double)s.lam[j - C * G] * s.c_slo;
        }
        tab[(long long)m * w + j] = cj;
        lmx = fmax(lmx, fabs(cj));
    }
    red_i[t] = bad ? 1 : 0;
    const double cmx = -block_min_d(-lmx, red_d);
    const int anybad = -block_min_i(-red_i[t], red_i);
    if (t == 0) sh_scale = cmx > 0.0 ? 1.0 / cmx : 1.0;
    __syncthreads();
    for (int j = t; j < nv; j += nt) tab[(long long)m * w + j] *= sh_scale;
    __syncthreads();

    int status = anybad ? 2 : 0;  // 0 optimal, 1 pivot limit, 2 infeasible start, 3 unbounded
    int pivots = 0, degenerate = 0;
    const double tol_d = 1e-12, tol_p = 1e-11;
    while (status == 0) {
        // entering column: the most negative reduced cost (lowest index on ties);
        // after a run of degenerate pivots, the lowest index with a negative
        // reduced cost (Bland's rule, which cannot cycle) until the objective moves
        const bool bland = degenerate >= kLpDegenerateRun;
        double dmin = 0.0;
        int cand = 0x7fffffff;
        for (int j = t; j < nv + m; j += nt) {
            if (j < C * G && z[j % G] <= 0) continue;
            const double d = tab[(long long)m * w + j];
            if (d < -tol_d && (bland ? cand == 0x7fffffff : d < dmin)) {
                dmin = d;
                cand = j;
            }
        }
        const int jin = block_min_key(bland ? 0.0 : dmin, cand, 0, wk_d, wk_i, wk_a).idx;
        if (jin == 0x7fffffff) break;  // optimal
        if (pivots >= max_pivots) {
            status = 1;
            break;
        }
        // ratio test: smallest b_i / a_ij over a_ij > 0, ties to the smallest basic index
        double best = INFINITY;
        int bb = 0x7fffffff, brow = -1;
        for (int r = t; r < m; r += nt) {
            const double a = tab[(long long)r * w + jin];
            if (a > tol_p) {
                const double q = tab[(long long)r * w + w - 1] / a;
                if (q < best || (q == best && basis[r] < bb)) {
                    best = q;
                    bb = basis[r];
                    brow = r;
                }
            }
        }
        const KeyIdx lv = block_min_key(best, bb, brow, wk_d, wk_i, wk_a);
        if (lv.idx == 0x7fffffff) {
            status = 3;
            break;
        }
        const int rsel = lv.aux;  // the row of the leaving basic variable
        degenerate = lv.key == 0.0 ? degenerate + 1 : 0;
        // pivot on (rsel, jin): each thread updates its own columns of every
        // row, reading eight rows before writing them back
        for (int r = t; r <= m; r += nt) col[r] = tab[(long long)r * w + jin];
        __syncthreads();
        const double piv = col[rsel];
        double *prow = tab + (long long)rsel * w;
        for (int j = t; j < w; j += nt) {
            const double pj = prow[j] / piv;
            prow[j] = pj;
            for (int r0 = 0; r0 <= m; r0 += 8) {
                double v[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const int r = r0 + q;
                    v[q] = r <= m ? tab[(long long)r * w + j] : 0.0;
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const int r = r0 + q;
                    if (r > m || r == rsel) continue;
                    const double f = col[r];
                    if (f != 0.0) tab[(long long)r * w + j] = v[q] - f * pj;
                }
            }
        }
        __syncthreads();
        if (t == 0) basis[rsel] = jin;
        __syncthreads();
        ++pivots;
    }
    // solution
    for (int j = t; j < C * G; j += nt) pi_out[j] = 0.0;
    __syncthreads();
    for (int r = t; r < m; r += nt) {
        const int j = basis[r];
        if (j < C * G) {
            const double v = tab[(long long)r * w + w - 1];
            pi_out[j] = v > 0.0 ? v : 0.0;
        }
    }
    __syncthreads();
    if (t == 0) {
        // objective of the routing: sum_c lam_c (sum_g pi_cg (W_c + c_gpu tau pp T - c_rej)
        // + c_slo s_c + c_rej) with s_c at its optimum max(0, sum_g pi_cg h_cg)
        double obj = 0.0;
        for (int c = 0; c < C; ++c) {
            double lin = 0.0, h = 0.0;
            for (int g = 0; g < G; ++g) {
                const double p = pi_out[c * G + g];
                if (z[g] <= 0) continue;
                lin = lin + p * (Wc[c] + s.c_gpu * (double)(s.tau[g] * s.pp[g]) * T[c * G + g] - s.c_rej);
                h = h + p * (Wq[g] + T[c * G + g] - (double)s.D[c]);
            }
            obj = obj + (double)s.lam[c] * (lin + s.c_slo * (h > 0.0 ? h : 0.0) + s.c_rej);
        }
        obj_out[0] = obj;
        info[0] = pivots;
        info[1] = status;
    }
}

// ------------------------------------------------------------------- LP2 ----
// The reservation sweep of the block step over a fixed W table: for c in
// order, the largest admissible grid point given the others, then the lowest
// argmin of W[c, 0..kmax], with 1e-6 tokens of slack on the bound so that a
// reservation at which the LP left the memory exactly full stays admissible.
// One block.  Incoming grid indices are clamped into [0, K).
__global__ __launch_bounds__(kSvcThreads) void sweep_kernel(
    const double *W, const int32_t *eta, int C, int K, int G, const double *conc,
    const double *cap, double kappa, const int32_t *k_in, int32_t *k_out, uint8_t *feasible)
{
    __shared__ double wk_d[kSvcThreads / 64];
    __shared__ int wk_i[kSvcThreads / 64], wk_a[kSvcThreads / 64];
    const int t = threadIdx.x, nt = blockDim.x;
    const double onek = 1.0 + kappa;
    for (int c = t; c < C; c += nt) k_out[c] = min(max(k_in[c], 0), K - 1);
    __syncthreads();
    for (int c = 0; c < C; ++c) {
        double bound = INFINITY;
        for (int g = t; g < G; g += nt) {
            const double cc = conc[c * G + g];
            if (!(cc > 0.0)) continue;
            double other = 0.0;
            for (int c2 = 0; c2 < C; ++c2)
                if (c2 != c) other = other + conc[c2 * G + g] * (double)eta[k_out[c2]];
            const double b = (cap[g] - onek * other) / (onek * cc);
            if (b < bound) bound = b;
        }
        bound = block_min_key(bound, 0, 0, wk_d, wk_i, wk_a).key;
        // largest k with eta[k] <= bound (eta ascending)
        int cand = -1;
        for (int kk = t; kk < K; kk += nt)
            if ((double)eta[kk] <= bound + kEtaSlack) cand = kk;
        const int kmax = -block_min_key(0.0, -cand, 0, wk_d, wk_i, wk_a).idx;
        const int hi = kmax < 0 ? 0 : kmax;
        // lowest argmin of W[c, 0..hi]
        const double *wr = W + (long long)c * K;
        double bv = INFINITY;
        int bk = 0x7fffffff;
        for (int kk = t; kk <= hi; kk += nt)
            if (wr[kk] < bv) {
                bv = wr[kk];
                bk = kk;
            }
        const int kbest = block_min_key(bv, bk, 0, wk_d, wk_i, wk_a).idx;
        if (t == 0) {
            k_out[c] = kbest;
            if (feasible) feasible[c] = kmax >= 0 ? 1 : 0;
        }
        __syncthreads();
    }
}

// Block 1 convergence: flag = (k_new == k && max |pi_new - pi| <= tol); then
// the new state becomes the current one.
__global__ __launch_bounds__(kSvcThreads) void converge_kernel(
    int C, int G, double tol, const int32_t *k_new, int32_t *k, const double *pi_new, double *pi,
    int32_t *flag)
{
    __shared__ double red_d[kSvcThreads];
    __shared__ int red_i[kSvcThreads];
    const int t = threadIdx.x, nt = blockDim.x;
    double d = 0.0;
    for (int i = t; i < C * G; i += nt) d = fmax(d, fabs(pi_new[i] - pi[i]));
    int same = 1;
    for (int c = t; c < C; c += nt) same &= k_new[c] == k[c];
    const double dmax = -block_min_d(-d, red_d);
    const int all_same = block_min_i(same, red_i);
    for (int i = t; i < C * G; i += nt) pi[i] = pi_new[i];
    for (int c = t; c < C; c += nt) k[c] = k_new[c];
    if (t == 0) flag[0] = (all_same && dmax <= tol) ? 1 : 0;
}

// --------------------------------------------------------------- Block 3 ----
// The objective at a given z with the routing, reservations and caching
// fixed, from per-class and per-configuration sums that do not depend on z.
struct ConfigPre {
    double *a, *gpu;                 // [C]
    double *used, *pre, *load, *X, *m2;  // [G]
    int32_t *route;                  // [G] some pi_cg > 0
};

__global__ void config_prep_kernel(SvcArgs s, const double *T, const double *ET2, const double *pi,
                                   const int32_t *eta_c, const uint8_t *delta, ConfigPre q)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int C = s.C, G = s.G;
    if (i < C) {
        const int c = i;
        double a = 0.0, gpu = 0.0;
        for (int g = 0; g < G; ++g) {
            const double p = pi[c * G + g];
            a = a + p;
            gpu = gpu + p * (s.c_gpu * (double)(s.tau[g] * s.pp[g]) * T[c * G + g]);
        }
        q.a[c] = a;
        q.gpu[c] = gpu;
    } else if (i < C + G) {
        const int g = i - C;
        double used = 0.0, pre = 0.0, load = 0.0, X = 0.0, m2 = 0.0;
        int route = 0;
        for (int c = 0; c < C; ++c) {
            const int j = c * G + g;
            const int dl = delta[j] ? s.Lpre[c] : 0;
            used = used + (double)s.lam[c] * T[j] * pi[j] * (double)(s.Lin[c] + eta_c[c] - dl);
            pre = pre + (double)dl;
            const double wgt = (double)s.lam[c] * pi[j];
            load = load + wgt * T[j];
            X = X + wgt;
            m2 = m2 + wgt * ET2[j];
            route |= pi[j] > 0.0;
        }
        q.used[g] = used;
        q.pre[g] = pre;
        q.load[g] = load;
        q.X[g] = X;
        q.m2[g] = m2;
        q.route[g] = route;
    }
}

constexpr int kMaxG = 32;

// objective at z (INFINITY when infeasible); zz holds z_g for g < G
__device__ double config_objective(const SvcArgs &s, const int32_t *zz, const double *Wc,
                                   const double *T, const double *pi, const ConfigPre &q)
{
    const int C = s.C, G = s.G;
    const double kap = 1.0 + s.kappa;
    double Wq[kMaxG];
#pragma unroll
    for (int g = 0; g < kMaxG; ++g) {
        Wq[g] = 0.0;
        if (g >= G) continue;
        if (zz[g] <= 0) {
            if (q.route[g]) return INFINITY;
            continue;
        }
        const double mem = kap * (q.used[g] / (double)zz[g]) + q.pre[g];
        if (!(mem <= s.u_max * (double)s.Mcap[g] * kMemSlack)) return INFINITY;
        if (q.X[g] > 0.0) {
            const double u = mem / (double)s.Mcap[g];
            const double tb = q.load[g] / q.X[g];
            const double cs2 = (q.m2[g] / q.X[g]) / (tb * tb) - 1.0;
            Wq[g] = u < 1.0 ? u * (1.0 + cs2) / (2.0 * (1.0 - u)) * tb : INFINITY;
        }
    }
    double obj = 0.0;
    for (int c = 0; c < C; ++c) {
        double resp = 0.0;
#pragma unroll
        for (int g = 0; g < kMaxG; ++g)
            if (g < G) resp = resp + pi[c * G + g] * (Wq[g] + T[c * G + g]);
        const double a = q.a[c];
        double sl = resp - a * (double)s.D[c];
        if (sl < 0.0) sl = 0.0;
        const double term = a * Wc[c] + q.gpu[c] + s.c_slo * sl + (1.0 - a) * s.c_rej;
        obj = obj + (double)s.lam[c] * term;
    }
    return obj;
}

// z of lexicographic rank r: ways[g][b] = number of (z_g..z_{G-1}) of cost <= b
__device__ void unrank(long long r, int G, int J, const int32_t *gpus, const long long *ways,
                       int32_t *zz)
{
    int b = J;
#pragma unroll
    for (int g = 0; g < kMaxG; ++g) {
        zz[g] = 0;
        if (g >= G) continue;
        int v = 0;
        while (v * gpus[g] <= b) {  // ends at a valid rank (r < ways[g][b]) or at the bound
            const long long cnt = ways[(long long)(g + 1) * (J + 1) + (b - v * gpus[g])];
            if (r < cnt) break;
            r -= cnt;
            ++v;
        }
        if (v * gpus[g] > b) v = b / gpus[g];
        zz[g] = v;
        b -= v * gpus[g];
    }
}

// One thread per rank; per block the lowest (objective, rank) and the number
// of feasible z.
__global__ __launch_bounds__(kSvcThreads) void config_search_kernel(
    SvcArgs s, long long nz, const int32_t *gpus, const long long *ways, const double *Wc,
    const double *T, const double *pi, ConfigPre q, double *part_obj, long long *part_rank,
    long long *part_feas)
{
    __shared__ double red_d[kSvcThreads];
    __shared__ long long red_l[kSvcThreads];
    const int t = threadIdx.x;
    const long long r = (long long)blockIdx.x * blockDim.x + t;
    double o = INFINITY;
    if (r < nz) {
        int32_t zz[kMaxG];
        unrank(r, s.G, s.J, gpus, ways, zz);
        o = config_objective(s, zz, Wc, T, pi, q);
    }
    const long long feas = o < INFINITY ? 1 : 0;
    red_l[t] = feas;
    __syncthreads();
    for (int w = kSvcThreads / 2; w > 0; w >>= 1) {
        if (t < w) red_l[t] += red_l[t + w];
        __syncthreads();
    }
    const long long nfeas = red_l[0];
    __syncthreads();
    const double omin = block_min_d(o, red_d);
    red_l[t] = (o == omin && o < INFINITY) ? r : 0x7fffffffffffffffLL;
    __syncthreads();
    for (int w = kSvcThreads / 2; w > 0; w >>= 1) {
        if (t < w && red_l[t + w] < red_l[t]) red_l[t] = red_l[t + w];
        __syncthreads();
    }
    if (t == 0) {
        part_obj[blockIdx.x] = omin;
        part_rank[blockIdx.x] = red_l[0];
        part_feas[blockIdx.x] = nfeas;
    }
}

// Final reduction over the blocks, the keep rule (the current z stays when it
// attains the minimum) and the change flag of the outer loop.
__global__ __launch_bounds__(kSvcThreads) void config_final_kernel(
    SvcArgs s, long long nparts, const double *part_obj, const long long *part_rank,
    const long long *part_feas, const int32_t *gpus, const long long *ways, const double *Wc,
    const double *T, const double *pi, ConfigPre q, int32_t *z, const uint8_t *delta_new,
    uint8_t *delta, double *best_obj, long long *best_rank, long long *n_feasible, int32_t *flag)
{
    __shared__ double red_d[kSvcThreads];
    __shared__ long long red_l[kSvcThreads];
    __shared__ int red_i[kSvcThreads];
    const int t = threadIdx.x, nt = blockDim.x;
    double o = INFINITY;
    long long rk = 0x7fffffffffffffffLL, nf = 0;
    for (long long p = t; p < nparts; p += nt) {
        nf += part_feas[p];
        const double v = part_obj[p];
        if (v < o || (v == o && part_rank[p] < rk)) {
            o = v;
            rk = part_rank[p];
        }
    }
    red_l[t] = nf;
    __syncthreads();
    for (int w = kSvcThreads / 2; w > 0; w >>= 1) {
        if (t < w) red_l[t] += red_l[t + w];
        __syncthreads();
    }
    const long long nfeas = red_l[0];
    __syncthreads();
    const double omin = block_min_d(o, red_d);
    red_l[t] = (o == omin) ? rk : 0x7fffffffffffffffLL;
    __syncthreads();
    for (int w = kSvcThreads / 2; w > 0; w >>= 1) {
        if (t < w && red_l[t + w] < red_l[t]) red_l[t] = red_l[t + w];
        __syncthreads();
    }
    const long long rmin = red_l[0];
    __syncthreads();
    // delta changes?
    int dchg = 0;
    if (delta_new && delta)
        for (int i = t; i < s.C * s.G; i += nt) dchg |= delta_new[i] != delta[i];
    const int anyd = -block_min_i(-dchg, red_i);
    if (t == 0) {
        int32_t zc[kMaxG], zb[kMaxG];
#pragma unroll
        for (int g = 0; g < kMaxG; ++g) zc[g] = g < s.G ? z[g] : 0;
        int zchg = 0;
        if (omin < INFINITY && rmin != 0x7fffffffffffffffLL) {
            unrank(rmin, s.G, s.J, gpus, ways, zb);
            const double ocur = config_objective(s, zc, Wc, T, pi, q);
            if (!(ocur == omin)) {
#pragma unroll
                for (int g = 0; g < kMaxG; ++g) {
                    if (g >= s.G) continue;
                    zchg |= zb[g] != zc[g];
                    z[g] = zb[g];
                }
            }
        }
        if (best_obj) best_obj[0] = omin;
        if (best_rank) best_rank[0] = omin < INFINITY ? rmin : -1;
        if (n_feasible) n_feasible[0] = nfeas;
        if (flag) flag[0] = (zchg || anyd) ? 1 : 0;
    }
    __syncthreads();
    if (delta_new && delta)
        for (int i = t; i < s.C * s.G; i += nt) delta[i] = delta_new[i];
}

// Objective of the current state (one thread).
__global__ void state_objective_kernel(SvcArgs s, const int32_t *z, const double *Wc,
                                       const double *T, const double *pi, ConfigPre q,
                                       double *out)
{
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        int32_t zc[kMaxG];
#pragma unroll
        for (int g = 0; g < kMaxG; ++g) zc[g] = g < s.G ? z[g] : 0;
        out[0] = config_objective(s, zc, Wc, T, pi, q);
    }
}

// ------------------------------------------------------------- launchers ----
hipError_t launch_service_times(const SvcArgs &s, const int64_t *count, const int64_t *sum,
                                const int64_t *sumsq, double *T, double *ET2, hipStream_t st)
{
    const int n = s.C * s.G;
    hipLaunchKernelGGL(service_times_kernel, dim3((n + 255) / 256), dim3(256), 0, st, s, count, sum,
                       sumsq, T, ET2);
    return hipGetLastError();
}

hipError_t launch_state(const SvcArgs &s, const double *T, const double *ET2, const double *pi,
                        const int32_t *z, const int32_t *eta_c, const uint8_t *delta, double *Wq,
                        double *cap, double *conc, double *mem, hipStream_t st)
{
    hipLaunchKernelGGL(state_kernel, dim3((s.G + 63) / 64), dim3(64), 0, st, s, T, ET2, pi, z,
                       eta_c, delta, Wq, cap, conc, mem);
    return hipGetLastError();
}

hipError_t launch_gather(const double *W, const int32_t *eta, const int32_t *k, int C, int K,
                         double *Wc, int32_t *eta_c, hipStream_t st)
{
    hipLaunchKernelGGL(gather_kernel, dim3((C + 255) / 256), dim3(256), 0, st, W, eta, k, C, K, Wc,
                       eta_c);
    return hipGetLastError();
}

hipError_t launch_cache(const double *conc, int n, uint8_t *delta, hipStream_t st)
{
    hipLaunchKernelGGL(cache_kernel, dim3((n + 255) / 256), dim3(256), 0, st, conc, n, delta);
    return hipGetLastError();
}

hipError_t launch_zero_u8(uint8_t *p, int n, hipStream_t st)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(zero_u8_kernel, dim3((n + 255) / 256), dim3(256), 0, st, p, n);
    return hipGetLastError();
}

constexpr size_t kLp1LdsBytes = 152 * 1024;  // dynamic LDS for the tableau (of 160 KB)

hipError_t lp1_prepare()
{
    return hipFuncSetAttribute(reinterpret_cast<const void *>(lp1_kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLp1LdsBytes);
}

size_t lp1_tableau_doubles(int C, int G)
{
    const long long nv = (long long)C * G + C, m = 2LL * C + G;
    return (size_t)((m + 1) * (nv + m + 1) + (m + 1));
}

hipError_t launch_lp1(const SvcArgs &s, const double *Wc, const double *T, const double *Wq,
                      const int32_t *z, const int32_t *eta_c, const uint8_t *delta, double *work,
                      int32_t *basis, int max_pivots, double *pi_out, double *obj_out,
                      int32_t *info, hipStream_t st)
{
    const long long nv = (long long)s.C * s.G + s.C, m = 2LL * s.C + s.G;
    double *tab = work, *col = work + (m + 1) * (nv + m + 1);
    // the tableau lives in LDS when it fits (one workgroup, every pivot touches all of it)
    const size_t bytes = lp1_tableau_doubles(s.C, s.G) * sizeof(double);
    const int in_lds = bytes <= kLp1LdsBytes ? 1 : 0;
    hipLaunchKernelGGL(lp1_kernel, dim3(1), dim3(kSvcThreads), in_lds ? bytes : 0, st, s, Wc, T,
                       Wq, z, eta_c, delta, tab, basis, col, in_lds, max_pivots, pi_out, obj_out,
                       info);
    return hipGetLastError();
}

hipError_t launch_sweep(const double *W, const int32_t *eta, int C, int K, int G,
                        const double *conc, const double *cap, double kappa, const int32_t *k_in,
                        int32_t *k_out, uint8_t *feasible, hipStream_t st)
{
    hipLaunchKernelGGL(sweep_kernel, dim3(1), dim3(kSvcThreads), 0, st, W, eta, C, K, G, conc, cap,
                       kappa, k_in, k_out, feasible);
    return hipGetLastError();
}

hipError_t launch_converge(int C, int G, double tol, const int32_t *k_new, int32_t *k,
                           const double *pi_new, double *pi, int32_t *flag, hipStream_t st)
{
    hipLaunchKernelGGL(converge_kernel, dim3(1), dim3(kSvcThreads), 0, st, C, G, tol, k_new, k,
                       pi_new, pi, flag);
    return hipGetLastError();
}

size_t config_pre_doubles(int C, int G) { return (size_t)(2 * C + 5 * G); }

static ConfigPre config_pre_view(double *d, int32_t *route, int C, int G)
{
    ConfigPre q;
    q.a = d;
    q.gpu = d + C;
    q.used = d + 2 * C;
    q.pre = q.used + G;
    q.load = q.pre + G;
    q.X = q.load + G;
    q.m2 = q.X + G;
    q.route = route;
    return q;
}

hipError_t launch_config_search(const SvcArgs &s, long long nz, const int32_t *gpus,
                                const long long *ways, const double *Wc, const double *T,
                                const double *ET2, const double *pi, const int32_t *eta_c,
                                const uint8_t *delta_eval, double *pre_d,
                                int32_t *pre_route, double *part_obj, long long *part_rank,
                                long long *part_feas, int32_t *z, const uint8_t *delta_new,
                                uint8_t *delta, double *best_obj, long long *best_rank,
                                long long *n_feasible, int32_t *flag, hipStream_t st)
{
    const ConfigPre q = config_pre_view(pre_d, pre_route, s.C, s.G);
    hipLaunchKernelGGL(config_prep_kernel, dim3((s.C + s.G + 255) / 256), dim3(256), 0, st, s, T,
                       ET2, pi, eta_c, delta_eval, q);
    const long long nb = (nz + kSvcThreads - 1) / kSvcThreads;
    hipLaunchKernelGGL(config_search_kernel, dim3((unsigned)nb), dim3(kSvcThreads), 0, st, s, nz,
                       gpus, ways, Wc, T, pi, q, part_obj, part_rank, part_feas);
    hipLaunchKernelGGL(config_final_kernel, dim3(1), dim3(kSvcThreads), 0, st, s, nb,
                       (const double *)part_obj, (const long long *)part_rank,
                       (const long long *)part_feas, gpus, ways, Wc, T, pi, q, z, delta_new, delta,
                       best_obj, best_rank, n_feasible, flag);
    return hipGetLastError();
}

hipError_t launch_state_objective(const SvcArgs &s, const double *T, const double *ET2,
                                  const double *pi, const int32_t *z, const int32_t *eta_c,
                                  const uint8_t *delta, const double *Wc, double *pre_d,
                                  int32_t *pre_route, double *out, hipStream_t st)
{
    const ConfigPre q = config_pre_view(pre_d, pre_route, s.C, s.G);
    hipLaunchKernelGGL(config_prep_kernel, dim3((s.C + s.G + 255) / 256), dim3(256), 0, st, s, T,
                       ET2, pi, eta_c, delta, q);
    hipLaunchKernelGGL(state_objective_kernel, dim3(1), dim3(64), 0, st, s, z, Wc, T, pi, q, out);
    return hipGetLastError();
}

}  // namespace dro
