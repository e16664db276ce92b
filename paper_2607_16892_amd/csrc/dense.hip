// Dense evaluation of the per-sample worst-case cost and its sums
// (paper, Appendix A, Step 4 closed form and Step 5 sums), plus the minimum
// over the multiplier grid (the Kantorovich dual of Appendix A, Step 3, with gamma on a grid).
//
// Work: one (class, grid point, multiplier, sample) term per evaluation,
// C * K * M * N_c terms in all.  This is max-plus arithmetic, not a dense
// contraction, so it runs on the fp32 VALU: every lane keeps a kTK x kTM
// register tile of (grid point, multiplier) accumulators and streams the
// samples of its class from LDS, where each tile of kTileN samples is staged
// once per block and read back as a wave-wide broadcast.
//
// Form of the term.  With B = c_w eta, C = c_p (L - eta), a1 = min(g, c_w) and
// a2 = min(g, c_p), the three candidates of Step 4 reduce, for 0 <= x, eta <= L,
// to the maximum of two lines (Q(eta, x) itself is the larger of c_w(eta - x)
// and c_p(x - eta), and for x, L - x >= 0 the smaller slope wins each pair):
//     phi = max(y1, y2),  y1 = B - a1 x,  y2 = C - a2 (L - x),
// which cross at x0 = (B - C + a2 L) / (a1 + a2).  Hence, exactly,
//     phi = y1 + (a1 + a2) relu(x - x0)      (used when c_w <= c_p)
//     phi = y2 + (a1 + a2) relu(x0 - x)      (used when c_w >  c_p)
// The line sums need only N and sum(x) of the slice and are formed in fp64;
// every (c, k, m, n) term still contributes its relu, evaluated per sample.
// The kink is measured from the grid point, x - x0 = (x - eta) - d with
// d = x0 - eta: x - eta is an exact integer formed once per (k, sample) and
// shared by the lane's kTM multipliers, and d is rounded to fp32 relative to
// its own size (it is 0, hence exact, for every lam >= max(c_p, c_w)).  The
// relu is then one instruction: u = +-(x - eta) 2^-16 plus -+d 2^-16 with the
// [0, 1] output clamp, exact while |x - x0| < 2^16 (x0 is clamped to
// [-1, L + 1], where relu is linear in the samples, and the clamped part is
// added back in the epilogue).  Choosing the side of the steeper line keeps
// the relu sum below twice the class's share of S, so the fp32 accumulation
// carries no cancellation.  Per evaluation the inner loop is
//     v_add_f32 t, u, a clamp ;  v_add_f32 acc, acc, t
// two fp32 VALU instructions that gfx950 issues at the double rate, plus one
// v_fma_f32 per (k, sample) shared by kTM evaluations.
//
// Accuracy: fp32 runs of kRun samples folded into fp64 in a fixed order, so
// the result is deterministic for a given launch plan.
#include "dro_internal.h"

namespace dro {

__device__ __forceinline__ int seg_of(const int32_t *seg, int c) { return seg ? seg[c] : c; }

// Crossing point of the two lines and the epilogue constants of one pair.
struct PairLines {
    double B, C, a1, a2, x0, x0c;
};

__device__ __forceinline__ PairLines pair_lines(float cp, float cw, float lam, int eta, int L)
{
    PairLines r;
    const float a1 = lam < cw ? lam : cw;
    const float a2 = lam < cp ? lam : cp;
    r.a1 = a1;
    r.a2 = a2;
    r.B = (double)cw * (double)eta;
    r.C = (double)cp * (double)(L - eta);
    r.x0 = (r.B - r.C + (double)a2 * (double)L) / ((double)a1 + (double)a2);
    r.x0c = r.x0 < -1.0 ? -1.0 : (r.x0 > (double)L + 1.0 ? (double)L + 1.0 : r.x0);
    return r;
}

__global__ __launch_bounds__(kThreads) void dense_kernel(DenseArgs a)
{
    __shared__ __attribute__((aligned(16))) float xs[kTileN];
    __shared__ long long red[kThreads];

    const DensePlan pl = a.plan;
    // Workgroups are dispatched to the XCDs in turn (block i to XCD i mod 8), so
    // XCD x is given one contiguous run of logical blocks; logical blocks that
    // read the same sample slice (one class and slice, every grid and multiplier
    // tile) are consecutive, so each slice is fetched into one XCD's L2.
    const long long nb = gridDim.x;
    const int xcd = (int)(blockIdx.x % kXcds);
    const long long q = nb / kXcds, r = nb % kXcds;
    long long b = xcd * q + min((long long)xcd, r) + blockIdx.x / kXcds;
    const int tm = (int)(b % pl.tiles_m);
    b /= pl.tiles_m;
    const int tk = (int)(b % pl.tiles_k);
    b /= pl.tiles_k;
    const int p = (int)(b % pl.P);
    b /= pl.P;
    const int c = (int)b;

    const int t = threadIdx.x;
    const int lm = t % pl.lanes_m, lk = t / pl.lanes_m;
    const int BK = kTK * pl.lanes_k, BM = kTM * pl.lanes_m;

    const int s = seg_of(a.seg, c);
    const long long n_beg = a.offsets[s], n_end = a.offsets[s + 1];
    const long long N = n_end - n_beg;
    const long long lo = n_beg + (N * p) / pl.P;
    const long long hi = n_beg + (N * (p + 1)) / pl.P;

    const float cp = a.c_p[c], cw = a.c_w[c];
    const int L = a.L[c];
    const bool upper = cw <= cp;                          // relu on x > x0
    const float sc = upper ? 0x1p-16f : -0x1p-16f;        // sign and scale of x - eta

    // grid point k_i = k0 + i * lanes_k, multiplier m_j = m0 + j * lanes_m
    // (recomputed where needed rather than held in registers)
    const int k0 = tk * BK + lk, m0 = tm * BM + lm;

    float eoff[kTK];        // -+eta 2^-16
    float add[kTK][kTM];    // -+(x0 - eta) 2^-16
#pragma unroll
    for (int i = 0; i < kTK; ++i) {
        const int eta = a.eta[min(k0 + i * pl.lanes_k, a.K - 1)];
        eoff[i] = -(float)eta * sc;
#pragma unroll
        for (int j = 0; j < kTM; ++j) {
            const PairLines q = pair_lines(cp, cw, a.lam[min(m0 + j * pl.lanes_m, a.M - 1)], eta, L);
            add[i][j] = -(float)(q.x0c - (double)eta) * sc;
        }
    }

    double acc64[kTK][kTM];
#pragma unroll
    for (int i = 0; i < kTK; ++i)
#pragma unroll
        for (int j = 0; j < kTM; ++j) acc64[i][j] = 0.0;

    long long xsum = 0;  // this thread's share of the slice's sample sum
    for (long long base = lo; base < hi; base += kTileN) {
        const int len = (int)min((long long)kTileN, hi - base);
        __syncthreads();
        for (int i = t; i < len; i += kThreads) {
            const int x = a.xi[base + i];
            xsum += x;
            xs[i] = (float)x;
        }
        __syncthreads();

        for (int u0 = 0; u0 < len; u0 += kRun) {
            const int cnt = min(kRun, len - u0);
            // the run's first sample initialises the accumulators
            float acc[kTK][kTM];
            auto first = [&](float x) {
#pragma unroll
                for (int i = 0; i < kTK; ++i) {
                    const float u = fmaf(x, sc, eoff[i]);
#pragma unroll
                    for (int j = 0; j < kTM; ++j)
                        acc[i][j] = __builtin_amdgcn_fmed3f(u + add[i][j], 0.0f, 1.0f);
                }
            };
            auto step = [&](float x) {
#pragma unroll
                for (int i = 0; i < kTK; ++i) {
                    const float u = fmaf(x, sc, eoff[i]);  // +-(x - eta) 2^-16, exact
#pragma unroll
                    for (int j = 0; j < kTM; ++j)
                        acc[i][j] += __builtin_amdgcn_fmed3f(u + add[i][j], 0.0f, 1.0f);
                }
            };

            first(xs[u0]);
            int u = 1;
            for (; u < 4 && u < cnt; ++u) step(xs[u0 + u]);
#pragma unroll 4
            for (; u + 4 <= cnt; u += 4) {
                const float4 x4 = *reinterpret_cast<const float4 *>(&xs[u0 + u]);
                step(x4.x);
                step(x4.y);
                step(x4.z);
                step(x4.w);
            }
            for (; u < cnt; ++u) step(xs[u0 + u]);

#pragma unroll
            for (int i = 0; i < kTK; ++i)
#pragma unroll
                for (int j = 0; j < kTM; ++j) acc64[i][j] += (double)acc[i][j];
        }
    }

    // slice sample sum (exact integer), shared by every pair of the block
    red[t] = xsum;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
        if (t < w) red[t] += red[t + w];
        __syncthreads();
    }
    const double sx = (double)red[0];
    const double n = (double)(hi - lo);

    // The epilogue recomputes the pair constants; hiding the indices from the
    // optimiser keeps it from holding the set-up values live across the loop.
    int k0e = k0, m0e = m0;
    asm volatile("" : "+v"(k0e), "+v"(m0e));

    double *out = a.out + ((long long)p * a.C + c) * (long long)a.K * a.M;
#pragma unroll
    for (int i = 0; i < kTK; ++i) {
        const int k = k0e + i * pl.lanes_k;
        if (k >= a.K) continue;
        const int eta = a.eta[k];
#pragma unroll
        for (int j = 0; j < kTM; ++j) {
            const int m = m0e + j * pl.lanes_m;
            if (m >= a.M) continue;
            const PairLines q = pair_lines(cp, cw, a.lam[m], eta, L);
            const double relu = acc64[i][j] * 65536.0;
            double line, corr = 0.0;
            if (upper) {
                line = n * q.B - q.a1 * sx;
                if (q.x0 < q.x0c) corr = n * (q.x0c - q.x0);
            } else {
                line = n * (q.C - q.a2 * (double)L) + q.a2 * sx;
                if (q.x0 > q.x0c) corr = n * (q.x0 - q.x0c);
            }
            out[(long long)k * a.M + m] = line + (q.a1 + q.a2) * (relu + corr);
        }
    }
}

int dense_blocks_per_cu()
{
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, dense_kernel, kThreads, 0) != hipSuccess || n < 1)
        n = 1;
    return n;
}

hipError_t launch_dense(const DenseArgs &a, hipStream_t st)
{
    hipLaunchKernelGGL(dense_kernel, dim3((unsigned)a.plan.blocks), dim3(kThreads), 0, st, a);
    return hipGetLastError();
}

__global__ void reduce_slices_kernel(const double *part, int P, long long n, double *S)
{
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    double acc = 0.0;
    for (int p = 0; p < P; ++p) acc += part[(long long)p * n + i];
    S[i] = acc;
}

hipError_t launch_reduce_slices(const double *part, int P, long long n, double *S, hipStream_t st)
{
    const long long blocks = (n + 255) / 256;
    hipLaunchKernelGGL(reduce_slices_kernel, dim3((unsigned)blocks), dim3(256), 0, st, part, P, n, S);
    return hipGetLastError();
}

// One thread per (c, k); radii in groups of 8 so S[c,k,:] is read E/8 times.
__global__ void min_over_lambda_kernel(const double *S, const int64_t *offsets, const int32_t *seg,
                                       const float *lam, const float *eps, int E, int C, int K,
                                       int M, double *W, int32_t *m_star)
{
    const long long ck = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (ck >= (long long)C * K) return;
    const int c = (int)(ck / K), k = (int)(ck % K);
    const int s = seg_of(seg, c);
    const double N = (double)(offsets[s + 1] - offsets[s]);
    const double *row = S + ck * M;
    for (int e0 = 0; e0 < E; e0 += 8) {
        double best[8];
        int bm[8];
        double ev[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            best[q] = __builtin_inf();
            bm[q] = 0;
            ev[q] = (e0 + q < E) ? (double)eps[(long long)(e0 + q) * C + c] : 0.0;
        }
        for (int m = 0; m < M; ++m) {
            const double lm = (double)lam[m];
            const double q_ = __ddiv_rn(row[m], N);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const double J = __dadd_rn(__dmul_rn(lm, ev[q]), q_);
                if (J < best[q]) {
                    best[q] = J;
                    bm[q] = m;
                }
            }
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (e0 + q >= E) break;
            const long long o = ((long long)(e0 + q) * C + c) * K + k;
            W[o] = best[q];
            if (m_star) m_star[o] = bm[q];
        }
    }
}

hipError_t launch_min_over_lambda(const double *S, const int64_t *offsets, const int32_t *seg,
                                  const float *lam, const float *eps, int E, int C, int K, int M,
                                  double *W, int32_t *m_star, hipStream_t st)
{
    const long long n = (long long)C * K;
    hipLaunchKernelGGL(min_over_lambda_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                       S, offsets, seg, lam, eps, E, C, K, M, W, m_star);
    return hipGetLastError();
}

}  // namespace dro
