// Dense evaluation of the per-sample worst-case cost and its sums
// (paper, Appendix A, Step 4 closed form and Step 5 sums), plus the minimum
// over the multiplier grid (eq. app_kantorovich with gamma on a grid).
//
// Work: one (class, grid point, multiplier, sample) term per evaluation,
// C * K * M * N_c terms in all.  This is max-plus arithmetic, not a dense
// contraction, so it runs on the fp32 VALU: every lane keeps a kTK x kTM
// register tile of (grid point, multiplier) accumulators and streams the
// samples of its class from LDS, where each tile of kTileN samples is
// staged once per block and read back as a wave-wide broadcast.
//
// Per sample x and grid point eta the lambda-independent parts are formed
// once and shared by the kTM multipliers of the lane:
//   A_p = c_p (x - eta),  A_w = c_w (eta - x),  A = max(A_p, A_w) = Q(eta, x)
// and per multiplier lam the two boundary candidates are
//   c_w eta - lam x           = A_w + (c_w - lam) x
//   c_p (L - eta) - lam (L-x) = A_p + (c_p - lam) (L - x)
// so that every rounded constant multiplies a quantity no larger than the
// candidate it feeds (the large constants c_w eta and c_p (L - eta) are never
// rounded on their own).  phi = max3(A, both candidates).
//
// Accuracy: fp32 runs of at most kRun samples are folded into fp64 in a fixed
// order, so the result is deterministic for a given launch plan.
#include "dro_internal.h"

namespace dro {

__device__ __forceinline__ int seg_of(const int32_t *seg, int c) { return seg ? seg[c] : c; }

__global__ __launch_bounds__(kThreads) void dense_kernel(DenseArgs a)
{
    __shared__ __attribute__((aligned(16))) float xs[kTileN];

    const DensePlan pl = a.plan;
    long long b = blockIdx.x;
    const int p = (int)(b % pl.P);
    b /= pl.P;
    const int tm = (int)(b % pl.tiles_m);
    b /= pl.tiles_m;
    const int tk = (int)(b % pl.tiles_k);
    b /= pl.tiles_k;
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
    const float Lf = (float)a.L[c];

    int kk[kTK], mm[kTM];
    float etaf[kTK], gw[kTM], gp[kTM];
#pragma unroll
    for (int i = 0; i < kTK; ++i) {
        kk[i] = tk * BK + lk + i * pl.lanes_k;
        etaf[i] = (float)a.eta[min(kk[i], a.K - 1)];
    }
#pragma unroll
    for (int j = 0; j < kTM; ++j) {
        mm[j] = tm * BM + lm + j * pl.lanes_m;
        const float lam = a.lam[min(mm[j], a.M - 1)];
        gw[j] = cw - lam;
        gp[j] = cp - lam;
    }

    double acc64[kTK][kTM];
#pragma unroll
    for (int i = 0; i < kTK; ++i)
#pragma unroll
        for (int j = 0; j < kTM; ++j) acc64[i][j] = 0.0;

    for (long long base = lo; base < hi; base += kTileN) {
        const int len = (int)min((long long)kTileN, hi - base);
        __syncthreads();
        for (int i = t; i < len; i += kThreads) xs[i] = (float)a.xi[base + i];
        __syncthreads();

        for (int u0 = 0; u0 < len; u0 += kRun) {
            const int cnt = min(kRun, len - u0);
            float acc[kTK][kTM];
#pragma unroll
            for (int i = 0; i < kTK; ++i)
#pragma unroll
                for (int j = 0; j < kTM; ++j) acc[i][j] = 0.0f;

            auto step = [&](float x) {
                const float lx = Lf - x;
#pragma unroll
                for (int i = 0; i < kTK; ++i) {
                    const float d = x - etaf[i];
                    const float Ap = cp * d;
                    const float Aw = -(cw * d);
                    const float A = fmaxf(Ap, Aw);
#pragma unroll
                    for (int j = 0; j < kTM; ++j) {
                        const float t0 = fmaf(gw[j], x, Aw);
                        const float tL = fmaf(gp[j], lx, Ap);
                        acc[i][j] += fmaxf(fmaxf(A, t0), tL);
                    }
                }
            };

            int u = 0;
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

    double *out = a.out + ((long long)p * a.C + c) * (long long)a.K * a.M;
#pragma unroll
    for (int i = 0; i < kTK; ++i) {
        if (kk[i] >= a.K) continue;
#pragma unroll
        for (int j = 0; j < kTM; ++j) {
            if (mm[j] >= a.M) continue;
            out[(long long)kk[i] * a.M + mm[j]] = acc64[i][j];
        }
    }
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
