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
// keeps kTM thresholds and 32-bit sums of one grid point.  Every
// kHalfSadSteps instructions the bit 2^31 of each sum moves into a 16-bit
// carry in LDS, so a sum spans any number of samples without a flush.
//
// Reduction and schedule.  Each tile's samples are split into P slices, and
// a persistent grid (every block resident) claims them with atomic counters:
// a block first drains its own tiles, then the tiles of its XCD with the most
// unclaimed slices, then any tile.  It keeps a tile's sums in registers over
// all the consecutive slices it claims of that tile and adds them to the
// [C][K][M] table with one 64-bit atomic per pair when it moves to another
// tile (a run).  Integer addition is associative, so the table does not
// depend on which block took which slice.  The wave arbiter of a compute unit
// favours its oldest waves, which would let one of its blocks finish its tiles
// far ahead of the others (and then take many short runs elsewhere); so at
// every claim a block sets its waves' issue priority from its lead over the
// average block, read from a counter of all claims.  Within a run, the claim
// of the next slice is issued when a slice starts and read when it ends.
#include <algorithm>

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
    // two staging buffers of kT samples (kT / kThreads prefetch registers per
    // lane); at the start of a run the same memory passes the tile's
    // thresholds from a rolled loop into registers
    constexpr int kT = 4096;
    __shared__ __attribute__((aligned(16))) uint16_t xs[kTileN];
    __shared__ uint16_t carry[kTM * kThreads];
    __shared__ int s_claim, s_prio;
    __shared__ int s_best[kThreads / 64], s_left[kThreads / 64];
    static_assert(kTileN >= kThreads * kTM, "the threshold table shares the sample buffers");
    static_assert(kT % kThreads == 0 && kT % 16 == 0 && 2 * kT <= kTileN, "staging shape");

    const DensePlan pl = a.plan;
    const int nb = (int)gridDim.x;
    const int T = a.C * pl.tiles;  // tile tau: class tau / tiles, tile tau % tiles of it
    // Workgroups are dispatched to the XCDs in turn (block i to XCD i mod 8), so
    // XCD x is given one contiguous run of logical blocks, whose own tiles are
    // one contiguous range [xt0, xt1): the blocks on an XCD read the samples of
    // a few classes, which stay in its L2.
    const int xcd = (int)(blockIdx.x % kXcds);
    const int qx = nb / kXcds, rx = nb % kXcds;
    const int xb0 = xcd * qx + min(xcd, rx);
    const int xb1 = xb0 + qx + (xcd < rx ? 1 : 0);
    const int b = xb0 + (int)(blockIdx.x / kXcds);
    auto own = [&](int lb) { return (int)(((long long)lb * T) / nb); };
    const int xt0 = own(xb0), xt1 = own(xb1);
    int next_own = own(b);
    const int own_end = own(b + 1);

    const int t = threadIdx.x;
    const int lm = t % pl.lanes_m, lk = t / pl.lanes_m;
    const int BM = kTM * pl.lanes_m;

    uint32_t thr[kTM];  // (t + 1) in both 16-bit halves
    uint32_t acc[kTM];
#pragma unroll
    for (int j = 0; j < kTM; ++j) {
        acc[j] = 0u;
        carry[j * kThreads + t] = 0;
    }
    int c = 0, k = 0, m0 = 0;
    // Sample codes 0 pad the end of a slice to whole groups of sixteen; each
    // adds t + 1 to a sum, which the flush takes off again.
    int pads = 0, steps = 0;

    auto normalize = [&]() {
        // (the address is hidden from the optimiser, which would otherwise keep
        // the 32 carry addresses live across the sample loop)
        int te = t;
        asm volatile("" : "+v"(te));
        uint16_t *cp = carry + te;
#pragma unroll
        for (int j = 0; j < kTM; ++j) {
            cp[j * kThreads] += (uint16_t)(acc[j] >> 31);
            acc[j] &= 0x7fffffffu;
        }
        steps = 0;
    };
    auto flush = [&]() {
        int ke = k, me = m0, ce = c, te = t;
        asm volatile("" : "+v"(ke), "+v"(me), "+v"(ce), "+v"(te));
        unsigned long long *row = a.R + ((long long)ce * a.K + ke) * a.M;
        uint16_t *cp = carry + te;
        if (ke < a.K) {
#pragma unroll
            for (int j = 0; j < kTM; ++j) {
                const int m = me + j * pl.lanes_m;
                uint32_t a32 = acc[j];
                asm volatile("" : "+v"(a32));  // keeps the sums 32-bit through the sample loop
                const unsigned long long tot = ((unsigned long long)cp[j * kThreads] << 31) + a32 -
                                               (unsigned long long)pads * (thr[j] & 0xffffu);
                if (m < a.M) atomicAdd(row + m, tot);
            }
        }
#pragma unroll
        for (int j = 0; j < kTM; ++j) {
            acc[j] = 0u;
            cp[j * kThreads] = 0;
        }
        pads = 0;
        steps = 0;
    };
    // the thresholds of tile tau (lanes past K or M take the last valid pair;
    // their sums are never stored)
    auto start_run = [&](int tau) {
        c = tau / pl.tiles;
        const int tile = tau % pl.tiles;
        const int tm = tile % pl.tiles_m, tk = tile / pl.tiles_m;
        k = tk * pl.lanes_k + lk;
        m0 = tm * BM + lm;
        const float cpf = a.c_p[c], cwf = a.c_w[c];
        const bool upper = cwf <= cpf;
        const int64_t CP = fix33(cpf), CW = fix33(cwf);
        const int L = a.L[c];
        const int eta = a.eta[min(k, a.K - 1)];
        // (four at a time: their multiplier loads overlap, and the 64-bit
        // arithmetic of four pairs fits beside the live sums)
#pragma unroll 4
        for (int j = 0; j < kTM; ++j) {
            const int m = min(m0 + j * pl.lanes_m, a.M - 1);
            const PairLinesFix q = pair_lines_fix(CP, CW, fix33(a.lam[m]), eta, L);
            xs[j * kThreads + t] = (uint16_t)(pair_kink(q, upper, L).tc + 1);
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kTM; ++j) thr[j] = (uint32_t)xs[j * kThreads + t] * 0x10001u;
        __syncthreads();
    };
    // The samples xi[lo, hi) in buffers of kT: the next buffer's samples are
    // loaded into registers while this one is evaluated, then stored; one
    // barrier per buffer.
    constexpr int kPer = kT / kThreads;
    int32_t pf[kPer];
    auto run_slice = [&](long long lo, long long hi) {
        auto fetch = [&](long long base) {
            // a block-uniform base and clamped 32-bit lane offsets: one
            // address register per load and no branches
            const int32_t *tp = a.xi + base;
            const int len = (int)min((long long)kT, hi - base);
#pragma unroll
            for (int r = 0; r < kPer; ++r) {
                const int i = t + r * kThreads;
                const int x = tp[min(i, len - 1)];
                pf[r] = i < len ? x : -1;
            }
        };
        auto put = [&](int buf) {
            uint16_t *dst = xs + buf * kT;
#pragma unroll
            for (int r = 0; r < kPer; ++r) dst[t + r * kThreads] = (uint16_t)(pf[r] + 1);
        };
        const int nbuf = (int)((hi - lo + kT - 1) / kT);
        if (nbuf > 0) {
            fetch(lo);
            put(0);
        }
        __syncthreads();
        for (int i = 0; i < nbuf; ++i) {
            const long long base = lo + (long long)i * kT;
            const int len = (int)min((long long)kT, hi - base);
            const int len16 = (len + 15) & ~15;
            if (steps + len16 / 2 > kHalfSadSteps) normalize();
            if (i + 1 < nbuf) fetch(base + kT);
            pads += len16 - len;
            steps += len16 / 2;
            // sixteen samples (two broadcast LDS reads) per step
            const uint4 *x4 = reinterpret_cast<const uint4 *>(xs + (i & 1) * kT);
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
            if (i + 1 < nbuf) put((i + 1) & 1);
            __syncthreads();
        }
    };
    // Issue priority from this block's lead over the average block: done is
    // the number of slices it has claimed, g the number all blocks had claimed
    // before its latest claim; 0 for a slice or more ahead, 3 for more than a
    // slice behind.
    int done = 0;
    auto prio_of = [&](long long g) {
        const long long lead = (long long)done * nb - g;  // in 1/nb slices
        return lead >= nb ? 0 : (lead >= 0 ? 1 : (lead >= -nb ? 2 : 3));
    };
    auto set_prio = [&](int level) {
        switch (level) {
        case 0: __builtin_amdgcn_s_setprio(0); break;
        case 1: __builtin_amdgcn_s_setprio(1); break;
        case 2: __builtin_amdgcn_s_setprio(2); break;
        default: __builtin_amdgcn_s_setprio(3); break;
        }
    };
    // Claims the next slice of tile tau for the whole block and waits for it
    // (block-uniform result: P or more means the tile is drained).
    auto claim = [&](int tau) {
        __syncthreads();
        if (t == 0) {
            s_claim = (int)atomicAdd(a.claim + tau, 1u);
            s_prio = prio_of((long long)atomicAdd(a.claim + T, 1u));
        }
        __syncthreads();
        return s_claim;
    };
    // The tile of [q0, q1) with the most unclaimed slices (-1 if none): every
    // thread reads some counters, then a block-wide maximum (ties to the
    // higher index).  Counters only grow, and the coherent reads see every
    // completed claim, so a block that finds a tile drained never picks it
    // again: the search ends.
    auto most_left = [&](int q0, int q1) {
        int best = -1, left = 0;
        for (int q = q0 + t; q < q1; q += kThreads) {
            const int r = pl.P - (int)__hip_atomic_load(a.claim + q, __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT);
            if (r > left) {
                left = r;
                best = q;
            }
        }
        for (int d = 32; d >= 1; d >>= 1) {
            const int ob = __shfl_xor(best, d, 64), ol = __shfl_xor(left, d, 64);
            if (ol > left || (ol == left && ob > best)) {
                left = ol;
                best = ob;
            }
        }
        __syncthreads();
        if ((t & 63) == 0) {
            s_best[t >> 6] = best;
            s_left[t >> 6] = left;
        }
        __syncthreads();
        if (t == 0) {
            int bb = s_best[0], bl = s_left[0];
            for (int w = 1; w < kThreads / 64; ++w)
                if (s_left[w] > bl || (s_left[w] == bl && s_best[w] > bb)) {
                    bl = s_left[w];
                    bb = s_best[w];
                }
            s_claim = bl > 0 ? bb : -1;
        }
        __syncthreads();
        return s_claim;
    };

    if (pl.direct) {
        // Small problems: the grid has a block per slice (slices of a tile on
        // consecutive logical blocks) and the hardware hands blocks to compute
        // units as they free up; no claims.
        const int tau = b / pl.P, p = b % pl.P;
        start_run(tau);
        const int sg = seg_of(a.seg, c);
        const long long n_beg = a.offsets[sg], N = a.offsets[sg + 1] - n_beg;
        run_slice(n_beg + slice_start(N, p, pl.P), n_beg + slice_start(N, p + 1, pl.P));
        flush();
        return;
    }

    // Runs: pick a tile and claim a slice of it; take its thresholds; evaluate
    // its slices while claims on it succeed; add the sums to the table.
    bool any_xcd = xt0 == 0 && xt1 == T;  // search every tile (this XCD's are drained)
    for (;;) {
        int tau = -1, p = pl.P;
        while (p >= pl.P) {
            if (next_own < own_end) {
                tau = next_own++;
            } else {
                tau = any_xcd ? most_left(0, T) : most_left(xt0, xt1);
                if (tau < 0) {
                    if (any_xcd) break;
                    any_xcd = true;
                    continue;
                }
            }
            p = claim(tau);
        }
        if (p >= pl.P) break;  // every slice has been claimed
        ++done;
        set_prio(s_prio);
        start_run(tau);
        const int sg = seg_of(a.seg, c);
        const long long n_beg = a.offsets[sg], N = a.offsets[sg + 1] - n_beg;
        for (;;) {
            run_slice(n_beg + slice_start(N, p, pl.P), n_beg + slice_start(N, p + 1, pl.P));
            p = claim(tau);
            if (p >= pl.P) break;
            ++done;
            set_prio(s_prio);
        }
        flush();
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

__global__ void zero_u64_u32_kernel(unsigned long long *p, long long n, uint32_t *q, long long nq)
{
    const long long m = n > nq ? n : nq;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < m;
         i += (long long)gridDim.x * blockDim.x) {
        if (i < n) p[i] = 0ull;
        if (i < nq) q[i] = 0u;
    }
}

hipError_t launch_zero_u64_u32(unsigned long long *p, long long n, uint32_t *q, long long nq,
                               hipStream_t st)
{
    const long long m = std::max(n, nq);
    if (m <= 0) return hipSuccess;
    hipLaunchKernelGGL(zero_u64_u32_kernel, dim3((unsigned)std::min((m + 255) / 256, kMaxGridBlocks)),
                       dim3(256), 0, st, p, n, q, nq);
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
__device__ __forceinline__ void dense_finish_one(const DenseFinishArgs &a, long long i)
{
    const long long KM = (long long)a.K * a.M;
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

__global__ void dense_finish_kernel(DenseFinishArgs a)
{
    const long long n = (long long)a.C * a.K * a.M;
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (long long)gridDim.x * blockDim.x)
        dense_finish_one(a, i);
}

hipError_t launch_dense_finish(const DenseFinishArgs &a, hipStream_t st)
{
    const long long n = (long long)a.C * a.K * a.M;
    hipLaunchKernelGGL(dense_finish_kernel, dim3((unsigned)std::min((n + 255) / 256, kMaxGridBlocks)),
                       dim3(256), 0, st, a);
    return hipGetLastError();
}

// One wave per (c, k) row.  The wave stages q_m = S[c,k,m] / N and lambda_m
// for a chunk of multipliers in LDS (coalesced reads of the row, each quotient
// computed once); then its 64 lanes split into g groups of 64/g, g the power of
// two covering E (at most 64), group j taking radius e0 + j and its lanes the
// multipliers m = part, part + 64/g, ... of the chunk.  Each lane keeps the
// smallest J of its multipliers (the lowest m among equal values, as it visits
// them in ascending order), then log2(64/g) shuffle steps take the smallest J
// of the group, ties to the lowest m: the same J bits and the same lowest m as
// a scan over m.
constexpr int kMinWaves = 4;    // waves (rows) per block
constexpr int kMinChunk = 256;  // multipliers staged per wave at a time

__global__ __launch_bounds__(64 * kMinWaves) void min_over_lambda_kernel(
    const double *S, const int64_t *offsets, const int32_t *seg, const float *lam, const float *eps,
    int E, int C, int K, int M, double *W, int32_t *m_star)
{
    __shared__ double2 st[kMinWaves][kMinChunk];  // (q_m, lambda_m)
    const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
    // rows in a grid-stride loop of whole waves (no block barrier below)
    for (long long ck = (long long)blockIdx.x * kMinWaves + w; ck < (long long)C * K;
         ck += (long long)gridDim.x * kMinWaves) {
        const int c = (int)(ck / K), k = (int)(ck % K);
        const int s = seg_of(seg, c);
        const double N = (double)(offsets[s + 1] - offsets[s]);
        const double *row = S + ck * M;
        int lg = 0;  // log2 of the groups
        while (lg < 6 && (1 << lg) < E) ++lg;
        const int lp = 6 - lg;  // log2 of the lanes per group
        const int part = lane & ((1 << lp) - 1), grp = lane >> lp;
        double2 *q = st[w];
        for (int e0 = 0; e0 < E; e0 += 1 << lg) {
            const int e = e0 + grp;
            const double ev = e < E ? (double)eps[(long long)e * C + c] : 0.0;
            double best = __builtin_inf();
            int bm = M;  // no multiplier yet: loses every comparison below
            for (int m0 = 0; m0 < M; m0 += kMinChunk) {
                const int mc = min(kMinChunk, M - m0);
                if (e0 == 0 || M > kMinChunk) {  // else the one chunk is still staged
                    __builtin_amdgcn_wave_barrier();  // the last chunk's reads come first
                    for (int i = lane; i < mc; i += 64)
                        q[i] = make_double2(__ddiv_rn(row[m0 + i], N), (double)lam[m0 + i]);
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                    __builtin_amdgcn_wave_barrier();
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
                }
                for (int i = part; i < mc; i += 1 << lp) {
                    const double2 v = q[i];
                    const double J = __dadd_rn(__dmul_rn(v.y, ev), v.x);
                    if (J < best) {
                        best = J;
                        bm = m0 + i;
                    }
                }
            }
            for (int d = (1 << lp) >> 1; d >= 1; d >>= 1) {
                const double ob = __shfl_xor(best, d, 64);
                const int om = __shfl_xor(bm, d, 64);
                if (ob < best || (ob == best && om < bm)) {
                    best = ob;
                    bm = om;
                }
            }
            if (part == 0 && e < E) {
                const long long o = ((long long)e * C + c) * K + k;
                W[o] = best;
                if (m_star) m_star[o] = bm;
            }
        }
    }
}

hipError_t launch_min_over_lambda(const double *S, const int64_t *offsets, const int32_t *seg,
                                  const float *lam, const float *eps, int E, int C, int K, int M,
                                  double *W, int32_t *m_star, hipStream_t st)
{
    const long long n = (long long)C * K;
    const long long blocks = std::min((n + kMinWaves - 1) / kMinWaves, kMaxGridBlocks);
    hipLaunchKernelGGL(min_over_lambda_kernel, dim3((unsigned)blocks),
                       dim3(64 * kMinWaves), 0, st, S, offsets, seg, lam, eps, E, C, K, M, W, m_star);
    return hipGetLastError();
}

}  // namespace dro
