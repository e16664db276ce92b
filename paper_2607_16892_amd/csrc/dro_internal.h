// Internal declarations shared by the HIP translation units of libdro.
// Not part of the public ABI (include/dro.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dro.h"

namespace dro {

// ---- dense evaluation -------------------------------------------------------
// Every lane owns one grid point and kTM multipliers; a 256-lane block covers a
// tile of lanes_k x (kTM * lanes_m) pairs of one class.  The samples of each
// tile are split into P slices.  A persistent grid of blocks claims slices
// (its own tiles first, then other tiles' unclaimed slices) and keeps a
// tile's sums in registers over consecutive slices of that tile.
constexpr int kThreads = 256;
constexpr int kTM = 32;
constexpr int kTileN = 8192;          // 16-bit LDS words of the staging buffers and the thresholds
constexpr int kHalfSadSteps = 32766;  // v_sad_u16 steps between carries: a sum kept below 2^31
                                      // takes 32766 more steps of at most 2 * 32770 below 2^32
constexpr int kXcds = 8;              // accelerator complex dies of one MI355X (one L2 each)

struct DensePlan {
    int lanes_m, lanes_k;  // lane grid inside a block
    int tiles_k, tiles_m;  // block tiles per class
    int tiles;             // tiles_k * tiles_m
    int P;                 // sample slices per tile
    int direct;            // 1: one block per slice, no claims (small problems)
    long long blocks;      // direct: C * tiles * P; else the persistent grid,
                           // min(resident blocks, C * tiles * P)
};

struct DenseArgs {
    const int64_t *offsets;
    const int32_t *seg;
    const int32_t *xi;
    const int32_t *L;
    const int32_t *eta;
    const float *lam;
    const float *c_p;
    const float *c_w;
    int C, K, M;
    DensePlan plan;
    unsigned long long *R;  // [C][K][M] sums of |x - t| over the class's samples, zeroed first
    uint32_t *claim;        // [C * tiles + 1] slice counters per tile, then the total; zeroed first
};

hipError_t launch_dense(const DenseArgs &a, hipStream_t st);
// resident dense blocks per compute unit (occupancy of dense_kernel)
int dense_blocks_per_cu();
// Launches whose block count grows with the problem loop over their items or
// rows with at most kMaxGridBlocks blocks, so a grid stays below 2^32
// work-items whatever the sizes.
constexpr long long kMaxGridBlocks = 1LL << 20;

// zeroes p[0, n) and q[0, nq)
hipError_t launch_zero_u64_u32(unsigned long long *p, long long n, uint32_t *q, long long nq,
                               hipStream_t st);

// S from the dense kernel's sums and the segments' prefix counts and sums
// (cnt, sum: [S][kHistBins], from launch_prefix), written over R as doubles.
struct DenseFinishArgs {
    const int64_t *offsets;
    const int32_t *seg;
    const int32_t *L;
    const int32_t *eta;
    const float *lam;
    const float *c_p;
    const float *c_w;
    const uint32_t *cnt;
    const uint64_t *sum;
    int C, K, M;
    unsigned long long *R;
};
hipError_t launch_dense_finish(const DenseFinishArgs &a, hipStream_t st);
// W[e,c,k] = min_m RN(RN(lam_m eps[e,c]) + RN(S[c,k,m] / N_c)), lowest m
hipError_t launch_min_over_lambda(const double *S, const int64_t *offsets, const int32_t *seg,
                                  const float *lam, const float *eps, int E, int C, int K, int M,
                                  double *W, int32_t *m_star, hipStream_t st);

// ---- quantile ----------------------------------------------------------------
constexpr int kHistBins = 32769;   // values 0 .. 2^15
hipError_t launch_fill_u32(uint32_t *p, long long n, uint32_t v, hipStream_t st);
// allows the histogram and quantile kernels their 128 KB of dynamic LDS (once per device)
hipError_t hist_prepare();
// blocks per segment for the histogram pass
int hist_parts(int S, long long max_seg, int num_cu);
// hist: [S][kHistBins], B blocks per segment (zeroed first when B > 1).
hipError_t launch_histogram(const int64_t *offsets, const int32_t *xi, int S, int B,
                            uint32_t *hist, hipStream_t st);
hipError_t launch_select(const int64_t *offsets, const int32_t *seg, const float *c_p,
                         const float *c_w, const uint32_t *hist, int C, int32_t *q_value,
                         int64_t *q_rank, hipStream_t st);

// ---- class_quantile (per-block packed histograms, then a select per class) ----
constexpr int kQTop = 32768;              // largest sample value, 2^15
constexpr int kQWords = kQTop / 2 + 1;    // packed 16-bit counts of the values 0 .. 2^15
constexpr int kQStride = kQWords + 3;     // words per stored row and LDS copy (16-byte multiple)
constexpr int kQBuckets = 256;            // coarse buckets of 128 values (the last also holds 2^15)
constexpr long long kQMaxPart = 65535;    // samples per block, so every 16-bit count fits
// blocks (parts) of a segment of n samples: about one block per compute unit
// over all S segments, each holding at most kQMaxPart samples
long long qhist_parts(int S, long long n, int num_cu);
// fine: [S][B][kQStride] u32, coarse: [S][B][kQBuckets] u32 (scratch, fully written)
// Parts: B per segment when boff is null (rows = S B), else boff[s] .. boff[s+1]
// are segment s's rows (device int64 [S+1], rows = boff[S]).
hipError_t launch_class_quantile(const int64_t *offsets, const int32_t *seg, const int32_t *xi,
                                 const float *c_p, const float *c_w, int S, int C, int B,
                                 const int64_t *boff, long long rows, uint32_t *fine,
                                 uint32_t *coarse, int32_t *q_value, int64_t *q_rank,
                                 hipStream_t st);

// ---- exact table (value counts and prefix sums) -------------------------------
// The prefix pass works in chunks of 4096 bins.  A sum array holds the S x
// kHistBins prefix sums followed by S x kPrefixChunks (count, sum) chunk totals
// that the pass uses as scratch: prefix_sum_words(S) u64 in all.
constexpr int kPrefixChunk = 4096;
constexpr int kPrefixChunks = (kHistBins + kPrefixChunk - 1) / kPrefixChunk;
inline size_t prefix_sum_words(int S)
{
    return (size_t)S * kHistBins + (size_t)S * kPrefixChunks * 2;
}
// cnt[s][v] = #{x <= v}, sum[s][v] = sum of the samples <= v of segment s, from
// its value histogram.
hipError_t launch_prefix(const uint32_t *hist, int S, uint32_t *cnt, uint64_t *sum, hipStream_t st);
// cnt: [S][kHistBins] u32, sum: prefix_sum_words(S) u64 scratch; k_star == null skips the argmin.
hipError_t launch_exact_table(const int64_t *offsets, const int32_t *seg, const int32_t *L,
                              const int32_t *eta, const float *lam, const float *c_p,
                              const float *c_w, const float *eps, const int32_t *k_max,
                              const uint32_t *hist, int S, int E, int C, int K, int M,
                              uint32_t *cnt, uint64_t *sum, double *W, int32_t *m_star,
                              int32_t *k_star, double *W_star, int32_t *m_at_star, hipStream_t st);
// Per (e, c): the lowest k <= k_max[c] (k_max may be null: K - 1) with the
// smallest W[e,c,k], W there, and m_star there (m_at_star may be null).
hipError_t launch_table_argmin(const double *W, const int32_t *m_star, const int32_t *k_max,
                               int E, int C, int K, int32_t *k_star, double *W_star,
                               int32_t *m_at_star, hipStream_t st);

// continuous-multiplier dual over the same prefix counts (gamma: the smallest minimiser)
hipError_t launch_continuous_dual(const int64_t *offsets, const int32_t *seg, const int32_t *L,
                                  const int32_t *eta, const float *c_p, const float *c_w,
                                  const float *eps, const uint32_t *hist, int S, int E, int C,
                                  int K, uint32_t *cnt, uint64_t *sum, double *W, double *gamma,
                                  hipStream_t st);

// ---- reservation cost and class moments ----------------------------------------
hipError_t launch_moments(const int32_t *seg, const uint32_t *hist, int C, int64_t *count,
                          int64_t *sum, int64_t *sumsq, int32_t *xmax, hipStream_t st);
hipError_t launch_reservation_cost(const int64_t *offsets, const int32_t *seg, const float *c_p,
                                   const float *c_w, const uint32_t *hist, int S, int C, int R,
                                   const int32_t *eta_r, uint32_t *cnt, uint64_t *sum,
                                   double *cost, int64_t *cover, hipStream_t st);

// ---- baseline reservations (policy comparison) ---------------------------------
constexpr int kMaxBaselineKs = 8;
struct BaselineKs {
    int n;                    // number of multiples k of the standard deviation
    int k[kMaxBaselineKs];    // each in [0, 64]
};
hipError_t launch_baselines(int C, const int64_t *count, const int64_t *sum, const int64_t *sumsq,
                            const int32_t *L, const BaselineKs &ks, const int32_t *q, int block,
                            int32_t *mean_r, int32_t *lp_r, int32_t *block_r, hipStream_t st);

// ---- block step ----------------------------------------------------------------
// sums: [C] scratch
hipError_t launch_bcd_init(const int64_t *offsets, const int32_t *seg, const int32_t *xi,
                           const int32_t *eta, int C, int K, long long max_n,
                           unsigned long long *sums, int32_t *k0, hipStream_t st);
// The block step's Gauss-Seidel sweep over the exact W [C][K] (one radius row),
// kcur [C] the state entering it (updated in place).
hipError_t launch_bcd_sweep(const double *W, const int32_t *eta, int C, int K, int G,
                            const float *cap, const float *conc, float kappa, int32_t *kcur,
                            int32_t *k_next, double *W_star, uint8_t *feasible, double *usage,
                            hipStream_t st);

// ---- serving model: routing LP, prefix caching, configuration search -------------
struct SvcArgs {
    int C, G;
    const int32_t *tau, *pp;
    const float *Mcap, *Cc, *Bc;
    const float *lam;
    const int32_t *Lin, *Lpre;
    const float *D;
    double alpha, beta, t_ar, NL, c_gpu, c_slo, c_rej, kappa, u_max;
    int J;
};

hipError_t launch_service_times(const SvcArgs &s, const int64_t *count, const int64_t *sum,
                                const int64_t *sumsq, double *T, double *ET2, hipStream_t st);
hipError_t launch_state(const SvcArgs &s, const double *T, const double *ET2, const double *pi,
                        const int32_t *z, const int32_t *eta_c, const uint8_t *delta, double *Wq,
                        double *cap, double *conc, double *mem, hipStream_t st);
hipError_t launch_gather(const double *W, const int32_t *eta, const int32_t *k, int C, int K,
                         double *Wc, int32_t *eta_c, hipStream_t st);
hipError_t launch_cache(const double *conc, int n, uint8_t *delta, hipStream_t st);
hipError_t launch_zero_u8(uint8_t *p, int n, hipStream_t st);
// doubles of the LP1 work area (tableau and pivot column)
size_t lp1_tableau_doubles(int C, int G);
// allow lp1_kernel its dynamic LDS (once per device)
hipError_t lp1_prepare();
hipError_t launch_lp1(const SvcArgs &s, const double *Wc, const double *T, const double *Wq,
                      const int32_t *z, const int32_t *eta_c, const uint8_t *delta, double *work,
                      int32_t *basis, int max_pivots, double *pi_out, double *obj_out,
                      int32_t *info, hipStream_t st);
hipError_t launch_sweep(const double *W, const int32_t *eta, int C, int K, int G,
                        const double *conc, const double *cap, double kappa, const int32_t *k_in,
                        int32_t *k_out, uint8_t *feasible, hipStream_t st);
hipError_t launch_converge(int C, int G, double tol, const int32_t *k_new, int32_t *k,
                           const double *pi_new, double *pi, int32_t *flag, hipStream_t st);
// doubles of the z-independent sums of the configuration search
size_t config_pre_doubles(int C, int G);
hipError_t launch_config_search(const SvcArgs &s, long long nz, const int32_t *gpus,
                                const long long *ways, const double *Wc, const double *T,
                                const double *ET2, const double *pi, const int32_t *eta_c,
                                const uint8_t *delta_eval, double *pre_d, int32_t *pre_route,
                                double *part_obj, long long *part_rank, long long *part_feas,
                                int32_t *z, const uint8_t *delta_new, uint8_t *delta,
                                double *best_obj, long long *best_rank, long long *n_feasible,
                                int32_t *flag, hipStream_t st);
hipError_t launch_state_objective(const SvcArgs &s, const double *T, const double *ET2,
                                  const double *pi, const int32_t *z, const int32_t *eta_c,
                                  const uint8_t *delta, const double *Wc, double *pre_d,
                                  int32_t *pre_route, double *out, hipStream_t st);

// ---- validation ----------------------------------------------------------------
hipError_t launch_seg_minmax(const int64_t *offsets, const int32_t *xi, int S, long long max_seg,
                             int32_t *mn, int32_t *mx, hipStream_t st);

}  // namespace dro
