// Dense evaluation of the per-sample worst-case cost and its sums
// (paper, Appendix A, Step 4 closed form and Step 5 sums), plus the minimum
// over the multiplier grid (the Kantorovich dual of Appendix A, Step 3, with
// gamma on a grid).
//
// Work: one (class, grid point, multiplier, sample) term per evaluation,
// C * K * M * N_c terms in all.  This is max-plus arithmetic, not a dense
// contraction, so it runs on the integer VALU; there is no MFMA.
//
// Form of the term.  In units of 2^-33 (fixed.h) the three candidates of
// Step 4 are the larger of two lines, y1 = B - A1 x and y2 = Cc - A2 (L - x),
// whose difference is y2 - y1 = De x - Nu.  With c_w <= c_p
//     phi = y1 + relu(De x - Nu),
// and with t = floor(Nu / De), r = Nu - De t in [0, De), for every integer x
//     relu(De x - Nu) = De relu(x - t) - r [x > t]
// (x > Nu / De exactly when x > t).  With c_w > c_p the mirror image holds
// around t = ceil(Nu / De): phi = y2 + De relu(t - x) - (De t - Nu) [x < t].
// Summed over a class's N samples,
//     S = sum y1 + De sum relu(x - t) - r #{x > t}
// and  sum relu(x - t) = (sum x - N t + sum |x - t|) / 2.
// The per-sample part of every term is |x - t|: that is what this kernel
// evaluates, once per (c, k, m, n).  The line sums need only N and sum x, and
// #{x > t} is one count per (c, k, m), read from the class's value counts in
// the epilogue; every piece is an integer, so S is exact and is rounded to
// double once.
//
// Instruction.  v_sad_u16 adds |a.lo - b.lo| + |a.hi - b.hi| (unsigned 16-bit
// halves) to a 32-bit accumulator: with two samples x + 1 packed in a and the
// threshold t + 1 in both halves of b, it evaluates two terms of one
// (k, m) pair in one single-rate VALU instruction.  Samples are staged in LDS
// as 16-bit x + 1 (x <= 2^15, t clamped to [-1, L] or [0, L + 1], so both
// fit), read back as wave-wide broadcasts of sixteen samples, and every lane
// keeps kTM thresholds and 32-bit sums of one grid point.  A 32-bit sum takes
// at most kMaxSadSteps instructions before it is added to the 64-bit table.
//
// Reduction.  The samples of a class are split into P slices with their own
// blocks; each block adds its exact integer sums to the [C][K][M] table with
// 64-bit atomics.  Integer addition is associative, so the result does not
// depend on the order the blocks finish in.
#include "dro_internal.h"
#include "fixed.h"

namespace dro {

__device__ __forceinline__ int seg_of(const int32_t *seg, int c) { return seg ? seg[c] : c; }

// Integer threshold t of a pair and its clamp to the range a 16-bit sample
// code can meet: [-1, L] when c_w <= c_p (relu(x - t)), [0, L + 1] otherwise
// (relu(t - x)).  Outside those ranges the sums are linear in the samples and
// the epilogue adds the difference.
struct Kink {
    int64_t t;
    int tc;
};

__device__ __forceinline__ Kink pair_kink(const PairLinesFix &q, bool upper, int L)
{
    Kink k;
    if (upper) {
        k.t = floor_div(q.Nu, q.De);
        k.tc = (int)(k.t < -1 ? -1 : (k.t > L ? L : k.t));
    } else {
        k.t = -floor_div(-q.Nu, q.De);
        k.tc = (int)(k.t < 0 ? 0 : (k.t > L + 1 ? L + 1 : k.t));
    }
    return k;
}

// First sample (relative to the segment start) of slice p of P: even offsets,
// so every slice but the last holds whole pairs of samples.
__device__ __forceinline__ long long slice_start(long long N, int p, int P)
{
    return p >= P ? N : 2 * ((N * p) / (2LL * P));
}

__global__ __launch_bounds__(kThreads) void dense_kernel(DenseArgs a)
{
    // The block's thresholds pass through LDS once (computed in a rolled loop),
    // then the same memory holds the sample tiles.
    __shared__ __attribute__((aligned(16))) uint16_t xs[kTileN];
    static_assert(kTileN >= kThreads * kTM, "the threshold table shares the sample tile");

    const DensePlan pl = a.plan;
    // Workgroups are dispatched to the XCDs in turn (block i to XCD i mod 8),
    // so XCD x is given one contiguous run of logical blocks.  Logical blocks
    // run through a class's tiles in groups of pl.group: all P slices of one
    // group, then the next group.  The blocks resident on an XCD at one time
    // then read a few sample slices and add into one group's part of the
    // table, which both stay in that XCD's L2.
    const long long nb = gridDim.x;
    const int xcd = (int)(blockIdx.x % kXcds);
    const long long qx = nb / kXcds, rx = nb % kXcds;
    long long b = xcd * qx + min((long long)xcd, rx) + blockIdx.x / kXcds;
    const long long per_class = (long long)pl.tiles * pl.P;
    const int c = (int)(b / per_class);
    long long rem = b % per_class;
    const int nfull = pl.tiles / pl.group;
    int tile, p;
    if (rem < (long long)nfull * pl.group * pl.P) {
        const int g = (int)(rem / ((long long)pl.group * pl.P));
        const int r2 = (int)(rem % ((long long)pl.group * pl.P));
        p = r2 / pl.group;
        tile = g * pl.group + r2 % pl.group;
    } else {
        const int r3 = (int)(rem - (long long)nfull * pl.group * pl.P);
        const int gl = pl.tiles - nfull * pl.group;
        p = r3 / gl;
        tile = nfull * pl.group + r3 % gl;
    }
    const int tm = tile % pl.tiles_m, tk = tile / pl.tiles_m;

    const int t = threadIdx.x;
    const int lm = t % pl.lanes_m, lk = t / pl.lanes_m;
    const int BM = kTM * pl.lanes_m;
    const int k = tk * pl.lanes_k + lk;  // one grid point per lane
    const int m0 = tm * BM + lm;         // multipliers m0 + j lanes_m

    const int s = seg_of(a.seg, c);
    const long long n_beg = a.offsets[s], N = a.offsets[s + 1] - n_beg;
    const long long lo = n_beg + slice_start(N, p, pl.P);
    const long long hi = n_beg + slice_start(N, p + 1, pl.P);

    const float cpf = a.c_p[c], cwf = a.c_w[c];
    const bool upper = cwf <= cpf;
    const int64_t CP = fix33(cpf), CW = fix33(cwf);
    const int L = a.L[c];
    const int eta = a.eta[min(k, a.K - 1)];

    for (int j = 0; j < kTM; ++j) {
        const int m = min(m0 + j * pl.lanes_m, a.M - 1);
        const PairLinesFix q = pair_lines_fix(CP, CW, fix33(a.lam[m]), eta, L);
        xs[j * kThreads + t] = (uint16_t)(pair_kink(q, upper, L).tc + 1);
    }
    __syncthreads();
    uint32_t thr[kTM];  // (t + 1) in both 16-bit halves
    uint32_t acc[kTM];
#pragma unroll
    for (int j = 0; j < kTM; ++j) {
        thr[j] = (uint32_t)xs[j * kThreads + t] * 0x10001u;
        acc[j] = 0u;
    }

    const bool row_ok = k < a.K;
    // Sample codes 0 pad the last tile to whole groups of sixteen; each adds
    // t + 1 to a sum, which the flush takes off again.
    int pads = 0, steps = 0;
    auto flush = [&]() {
        // Hiding the indices from the optimiser keeps it from holding the 32
        // table addresses live across the sample loop.
        int ke = k, me = m0;
        asm volatile("" : "+v"(ke), "+v"(me));
        unsigned long long *row = a.R + ((long long)c * a.K + ke) * a.M;
        if (row_ok) {
#pragma unroll
            for (int j = 0; j < kTM; ++j) {
                const int m = me + j * pl.lanes_m;
                if (m < a.M)
                    atomicAdd(row + m, (unsigned long long)(acc[j] - (uint32_t)pads * (thr[j] & 0xffffu)));
            }
        }
#pragma unroll
        for (int j = 0; j < kTM; ++j) acc[j] = 0u;
        pads = 0;
        steps = 0;
    };

    const uint4 *x4 = reinterpret_cast<const uint4 *>(xs);
    for (long long base = lo; base < hi; base += kTileN) {
        const int len = (int)min((long long)kTileN, hi - base);
        const int len16 = (len + 15) & ~15;
        if (steps + len16 / 2 > kMaxSadSteps) flush();
        __syncthreads();
        for (int i = t; i < len16; i += kThreads)
            xs[i] = i < len ? (uint16_t)(a.xi[base + i] + 1) : (uint16_t)0;
        __syncthreads();
        pads += len16 - len;
        steps += len16 / 2;

        // sixteen samples (two broadcast LDS reads) per step
        const int n8 = len16 / 16;
        for (int w = 0; w < n8; ++w) {
            const uint4 v = x4[2 * w], u = x4[2 * w + 1];
#pragma unroll
            for (int j = 0; j < kTM; ++j) acc[j] = __builtin_amdgcn_sad_u16(v.x, thr[j], acc[j]);
#pragma unroll
            for (int j = 0; j < kTM; ++j) acc[j] = __builtin_amdgcn_sad_u16(v.y, thr[j], acc[j]);
#pragma unroll
            for (int j = 0; j < kTM; ++j) acc[j] = __builtin_amdgcn_sad_u16(v.z, thr[j], acc[j]);
#pragma unroll
            for (int j = 0; j < kTM; ++j) acc[j] = __builtin_amdgcn_sad_u16(v.w, thr[j], acc[j]);
#pragma unroll
            for (int j = 0; j < kTM; ++j) acc[j] = __builtin_amdgcn_sad_u16(u.x, thr[j], acc[j]);
#pragma unroll
            for (int j = 0; j < kTM; ++j) acc[j] = __builtin_amdgcn_sad_u16(u.y, thr[j], acc[j]);
#pragma unroll
            for (int j = 0; j < kTM; ++j) acc[j] = __builtin_amdgcn_sad_u16(u.z, thr[j], acc[j]);
#pragma unroll
            for (int j = 0; j < kTM; ++j) acc[j] = __builtin_amdgcn_sad_u16(u.w, thr[j], acc[j]);
        }
    }
    if (steps > 0) flush();
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

__global__ void fill_u64_kernel(unsigned long long *p, long long n)
{
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0ull;
}

hipError_t launch_zero_u64(unsigned long long *p, long long n, hipStream_t st)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u64_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n);
    return hipGetLastError();
}

// #{x <= v} of a segment from its prefix counts (cn[v], v in [0, 2^15]).
__device__ __forceinline__ long long count_le(const uint32_t *cn, long long v, long long N)
{
    if (v < 0) return 0;
    if (v >= kHistBins - 1) return N;
    return (long long)cn[v];
}

// S[c,k,m] from the per-sample sums sum |x - t_c| of the dense kernel (in R,
// overwritten in place), the segment's value counts and its sample sum:
// exactly, in 128-bit integers in units of 2^-33, then rounded to double once.
__global__ void dense_finish_kernel(DenseFinishArgs a)
{
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    const long long KM = (long long)a.K * a.M;
    if (i >= (long long)a.C * KM) return;
    const int c = (int)(i / KM);
    const int k = (int)((i / a.M) % a.K);
    const int m = (int)(i % a.M);
    const int s = seg_of(a.seg, c);
    const long long N = a.offsets[s + 1] - a.offsets[s];
    const uint32_t *cn = a.cnt + (long long)s * kHistBins;
    const __int128 sx = (__int128)a.sum[(long long)s * kHistBins + kHistBins - 1];
    const float cpf = a.c_p[c], cwf = a.c_w[c];
    const bool upper = cwf <= cpf;
    const int L = a.L[c];
    const PairLinesFix q = pair_lines_fix(fix33(cpf), fix33(cwf), fix33(a.lam[m]), a.eta[k], L);
    const Kink kk = pair_kink(q, upper, L);
    const __int128 sad = (__int128)a.R[i];
    const __int128 n = N, tc = kk.tc, tt = kk.t;
    __int128 S;
    if (upper) {
        // sum relu(x - t) with the clamp undone for t < -1 (every sample above t)
        const __int128 Rt = (sx - n * tc + sad) / 2 + n * (tc > tt ? tc - tt : 0);
        const __int128 r = (__int128)q.Nu - (__int128)q.De * tt;
        const __int128 above = n - count_le(cn, kk.t, N);
        S = n * q.B - (__int128)q.A1 * sx + (__int128)q.De * Rt - r * above;
    } else {
        // sum relu(t - x) with the clamp undone for t > L + 1 (every sample below t)
        const __int128 Rt = (n * tc - sx + sad) / 2 + n * (tt > tc ? tt - tc : 0);
        const __int128 r = (__int128)q.De * tt - (__int128)q.Nu;
        const __int128 below = count_le(cn, kk.t - 1, N);
        S = n * ((__int128)q.Cc - (__int128)q.A2 * L) + (__int128)q.A2 * sx + (__int128)q.De * Rt -
            r * below;
    }
    reinterpret_cast<double *>(a.R)[i] = sfix128_to_double(S);
}

hipError_t launch_dense_finish(const DenseFinishArgs &a, hipStream_t st)
{
    const long long n = (long long)a.C * a.K * a.M;
    hipLaunchKernelGGL(dense_finish_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, a);
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
