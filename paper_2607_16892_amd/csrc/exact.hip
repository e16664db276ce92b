// Exact parts of the reservation path: the value histograms and prefix sums,
// the exact table (F1) and the argmin over an exact W table, the
// critical-fractile quantile, the block-step sweep and device-data checks.
//
// Compiled with -ffp-contract=off: every double expression below is the
// round-to-nearest-even sequence written, with no fused multiply-add.
//
// Fixed point.  Inside the library's limits (integers <= 2^15, binary32
// coefficients in [2^-10, 2^7]) every candidate of phi (Appendix A, Step 4)
// is an integer multiple of 2^-33 below 2^56, so phi is evaluated exactly in
// 64-bit integers and summed exactly in 128-bit integers.  The reported value
// is J = RN(RN(lam eps) + RN(RN(S) / N)) with RN(S) the correctly rounded
// double of the exact sum.
#include <algorithm>

#include "dro_internal.h"
#include "fixed.h"

namespace dro {

__device__ __forceinline__ int seg_of_x(const int32_t *seg, int c) { return seg ? seg[c] : c; }

#define HIPRET(expr)                                 \
    do {                                             \
        const hipError_t e_ = (expr);                \
        if (e_ != hipSuccess) return e_;             \
    } while (0)

// Exact S of one (class, grid point, multiplier), in units of 2^-33, from the
// prefix counts cn[v] = #{x <= v} and sums sm[v] = sum{x : x <= v} of the
// class's segment (N samples).  For 0 <= x, eta <= L the three candidates of
// Step 4 reduce to the larger of two lines, B - a1 x and C - a2 (L - x) with
// B = c_w eta, C = c_p (L - eta), a1 = min(g, c_w), a2 = min(g, c_p); the
// first is the larger up to t = floor((B - C + a2 L) / (a1 + a2)), so
//   S = B cnt(t) - a1 sum(t) + (C - a2 L)(N - cnt(t)) + a2 (sum_all - sum(t)),
// every term an exact integer (the sum is non-negative, as phi is).
__device__ __forceinline__ unsigned __int128 exact_S_prefix(const uint32_t *cn, const uint64_t *sm,
                                                           int64_t N, int64_t L, int64_t eta,
                                                           int64_t CP, int64_t CW, int64_t G)
{
    const int64_t B = CW * eta, Cc = CP * (L - eta);
    const int64_t A1 = G < CW ? G : CW, A2 = G < CP ? G : CP;
    const int64_t tmax = L < kHistBins - 1 ? L : kHistBins - 1;
    int64_t tt = floor_div(B - Cc + A2 * L, A1 + A2);
    tt = tt < -1 ? -1 : (tt > tmax ? tmax : tt);
    const __int128 ct = tt >= 0 ? (__int128)cn[tt] : 0;
    const __int128 st = tt >= 0 ? (__int128)sm[tt] : 0;
    const __int128 sum_all = (__int128)sm[kHistBins - 1];
    const __int128 S = (__int128)B * ct - (__int128)A1 * st + (__int128)(Cc - A2 * L) * ((__int128)N - ct) +
                       (__int128)A2 * (sum_all - st);
    return (unsigned __int128)S;
}

__global__ void fill_u32_kernel(uint32_t *p, long long n, uint32_t v)
{
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (long long)gridDim.x * blockDim.x)
        p[i] = v;
}

// -------------------------------------------------------------- quantile ----
hipError_t launch_fill_u32(uint32_t *p, long long n, uint32_t v, hipStream_t st)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)std::min((n + 255) / 256, kMaxGridBlocks)),
                       dim3(256), 0, st, p, n, v);
    return hipGetLastError();
}

// Calls count(x) for every sample of xi[lo, hi) handed to this thread of a
// kThreadsT-thread block: an unaligned head (up to the first 16-byte aligned
// address), a 16-byte body and a tail.  In the body every thread keeps eight
// 16-byte loads in flight, in two register sets of four: the next round's
// loads are issued before this round's samples are counted.  Body vector i
// goes to thread i mod kThreadsT, so even and odd threads see alternate
// vectors.  prologue() (block-wide: every thread calls it) runs once the
// first four loads are in flight and before any count, so the block's set-up
// (clearing its LDS counts) overlaps their latency.
template <int kThreadsT, class F, class G>
__device__ __forceinline__ void for_each_sample(const int32_t *xi, long long lo, long long hi, F &&count,
                                                G &&prologue)
{
    const int t = threadIdx.x;
    const long long mis = (long long)((reinterpret_cast<uintptr_t>(xi + lo) >> 2) & 3u);
    const long long a0 = min(hi, lo + ((4 - mis) & 3));
    const long long a1 = a0 + ((hi - a0) & ~3LL);
    const int4 *v4 = reinterpret_cast<const int4 *>(xi + a0);
    const long long nv = (a1 - a0) / 4;
    constexpr long long kRound = 4LL * kThreadsT;
    int4 qa[4], qb[4];
    // (unconditional loads, clamped to the last vector, so all four issue
    // back to back; tally skips the ones past the end)
    auto load = [&](long long r0, int4 (&d)[4]) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const long long i = r0 + r * kThreadsT + t;
            d[r] = v4[i < nv ? i : nv - 1];
        }
    };
    auto tally = [&](long long r0, const int4 (&d)[4]) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            if (r0 + r * kThreadsT + t >= nv) continue;
            count(d[r].x);
            count(d[r].y);
            count(d[r].z);
            count(d[r].w);
        }
    };
    if (nv > 0) load(0, qa);
    prologue();
    for (long long n = lo + t; n < a0; n += kThreadsT) count(xi[n]);
    for (long long r0 = 0; r0 < nv; r0 += 2 * kRound) {
        load(r0 + kRound, qb);
        tally(r0, qa);
        load(r0 + 2 * kRound, qa);
        tally(r0 + kRound, qb);
    }
    for (long long n = a1 + t; n < hi; n += kThreadsT) count(xi[n]);
}

// Block (segment s, part b of B): a private 32-bit LDS histogram of the values
// 0 .. 2^15 (128 KB) over its 1/B share of the segment, then added into the
// segment's histogram: with plain stores when the block covers the whole
// segment (B == 1), else with one atomic add per non-zero bin into a histogram
// the launch has zeroed (integer adds, so the result does not depend on the
// order).  Only the distinct values of a block cost a global access: about
// 7,800 of the 32,769 bins for a block of 62,500 heavy-tailed lengths.
constexpr int kHistThreads = 1024;

__global__ __launch_bounds__(kHistThreads) void histogram_kernel(const int64_t *offsets,
                                                                 const int32_t *xi, int B,
                                                                 uint32_t *hist)
{
    extern __shared__ uint32_t h[];  // kHistBins words
    const int s = (int)(blockIdx.x / B), b = (int)(blockIdx.x % B);
    const long long n0 = offsets[s], N = offsets[s + 1] - n0;
    const long long lo = n0 + (N * b) / B, hi = n0 + (N * (b + 1)) / B;
    const int t = threadIdx.x;
    for_each_sample<kHistThreads>(
        xi, lo, hi,
        [&](int v) {
            v = v < 0 ? 0 : (v > kHistBins - 1 ? kHistBins - 1 : v);
            atomicAdd(&h[v], 1u);
        },
        [&] {
            for (int i = t; i < kHistBins; i += kHistThreads) h[i] = 0;
            __syncthreads();
        });
    __syncthreads();
    uint32_t *o = hist + (long long)s * kHistBins;
    if (B == 1) {
        for (int i = t; i < kHistBins; i += kHistThreads) o[i] = h[i];
    } else {
        for (int i = t; i < kHistBins; i += kHistThreads) {
            const uint32_t c = h[i];
            if (c) atomicAdd(o + i, c);
        }
    }
}

__device__ int64_t exact_rank(float cp, float cw, int64_t N);

// ---- class_quantile: per-block histograms, then one select per class ----
//
// Block for row r (segment s, part b of its B_s parts, at most kQMaxPart
// samples; rows in a block-uniform loop) counts its share in LDS with 16-bit
// counts packed two to a word (value v < 2^15 in word v mod 2^14, low half
// for v < 2^14, high half above; 2^15 in the low half of word 2^14), in two
// copies: even threads add into one, odd threads into the other, which halves
// the lanes of one wave that meet on one LDS word when short lengths repeat.
// It then stores the two copies' sum (every count fits 16 bits, as the block
// holds at most 65,535 samples) with 16-byte non-temporal stores, as only the
// select reads it, once (on mixture-16x1M 1.4 us less per launch than plain
// stores), and, in the same pass, its counts per coarse bucket of 128 values.
// Segment s owns rows s B .. s B + B - 1 when every segment has B parts, else
// rows boff[s] .. boff[s + 1] - 1 of a table built by the host, in which the
// block finds its segment by bisection.  No global atomics: the select reads
// the segment's rows of the bucket it needs.
constexpr int kQThreads = 1024;
typedef uint32_t u32x4_nt __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kQThreads) void qhist_kernel(const int64_t *offsets, const int32_t *xi,
                                                          int S, int B, const int64_t *boff,
                                                          long long rows, uint32_t *fine,
                                                          uint32_t *coarse)
{
    extern __shared__ uint32_t h[];  // 2 x kQStride words
    const int t = threadIdx.x;
    for (long long r = blockIdx.x; r < rows; r += gridDim.x) {
        int s;
        long long b, Bs;
        if (boff) {  // the segment whose rows hold r: boff[s] <= r < boff[s + 1]
            int a = 0, z = S;
            while (z - a > 1) {
                const int mid = (a + z) >> 1;
                if (boff[mid] <= r) a = mid;
                else z = mid;
            }
            s = a;
            b = r - boff[s];
            Bs = boff[s + 1] - boff[s];
        } else {
            s = (int)(r / B);
            b = r % B;
            Bs = B;
        }
        const long long n0 = offsets[s], N = offsets[s + 1] - n0;
        const long long lo = n0 + (N * b) / Bs, hi = n0 + (N * (b + 1)) / Bs;
        uint32_t *hc = h + (t & 1) * kQStride;
        uint4 *h4 = reinterpret_cast<uint4 *>(h);
        const uint4 *g4 = reinterpret_cast<const uint4 *>(h + kQStride);
        for_each_sample<kQThreads>(
            xi, lo, hi,
            [&](int v) {
                v = v < 0 ? 0 : (v > kQTop ? kQTop : v);
                // bit 14 of v selects the half (v = 2^15 has it clear)
                atomicAdd(&hc[v < kQTop ? (v & (kQTop / 2 - 1)) : kQTop / 2], 1u << ((v >> 10) & 16));
            },
            [&] {
                for (int i = t; i < 2 * kQStride / 4; i += kQThreads) h4[i] = make_uint4(0u, 0u, 0u, 0u);
                __syncthreads();
            });
        __syncthreads();
        // 16-byte word group q = t + 1024 i (i < 4) holds the words 4q .. 4q + 3:
        // the values of coarse bucket q / 32 in its low halves and of bucket
        // 128 + q / 32 in its high halves, so the 32 lanes t mod 32 = 0 .. 31 of a
        // half-wave share both buckets.  The packed words add as plain 32-bit
        // integers: no sum of low halves exceeds the block's 65,535 samples.
        static_assert(kQThreads * 16 == kQTop / 2, "four word groups per thread");
        static_assert(kQStride % 4 == 0 && kQStride >= kQTop / 2 + 4, "row of whole word groups");
        uint4 *out = reinterpret_cast<uint4 *>(fine + r * kQStride);
        uint32_t *co = coarse + r * kQBuckets;
    #pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int q = t + kQThreads * i;
            const uint4 x = h4[q], y = g4[q];
            const uint4 c = make_uint4(x.x + y.x, x.y + y.y, x.z + y.z, x.w + y.w);
            __builtin_nontemporal_store(u32x4_nt{c.x, c.y, c.z, c.w}, reinterpret_cast<u32x4_nt *>(out + q));
            uint32_t p = (c.x + c.y) + (c.z + c.w);
            for (int d = 1; d < 32; d <<= 1) p += __shfl_xor(p, d, 64);
            if ((t & 31) == 0) {
                const int bk = q >> 5;
                co[bk] = p & 0xffffu;
                // the last bucket also holds the value 2^15
                co[128 + bk] = (p >> 16) + (bk == 127 ? (h[kQTop / 2] + h[kQStride + kQTop / 2]) & 0xffffu : 0u);
            }
        }
        if (t == 0) {  // the group of the value 2^15 and the padding words
            const uint4 x = h4[kQTop / 8], y = g4[kQTop / 8];
            out[kQTop / 8] = make_uint4(x.x + y.x, x.y + y.y, x.z + y.z, x.w + y.w);
        }
        __syncthreads();  // the next row clears the counts this row has read
    }
}

// Class c (segment s, its B rows at s B0 or boff[s]; classes in a
// block-uniform loop): the coarse counts of the rows summed per bucket, the
// bucket holding the exact rank j, then the counts of its values summed over
// the rows, and the value where the cumulative count reaches j.  Every thread
// issues its share of the rows' loads together.
__device__ void qselect_class(const int64_t *offsets, const int32_t *seg, const float *c_p,
                              const float *c_w, const uint32_t *fine, const uint32_t *coarse, int B0,
                              const int64_t *boff, int c, int32_t *q_value, int64_t *q_rank)
{
    constexpr int kG = kQThreads / kQBuckets;  // row groups of the coarse sum
    constexpr int kF = 129;                    // values of a bucket (the last adds 2^15)
    constexpr int kFG = kQThreads / 128;       // row groups of the fine sum
    __shared__ uint32_t part[kG][kQBuckets];
    __shared__ uint32_t fpart[kFG][kF];
    __shared__ uint32_t wsum[kQBuckets / 64];
    __shared__ int sel;
    __shared__ long long sel_below;
    __shared__ int64_t s_off[2], s_rank;
    __shared__ float s_cost[2];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int s = seg_of_x(seg, c);
    // the rank's inputs, loaded by every thread from addresses that differ by
    // lane: vector loads in flight with the coarse loads below, not waited for
    // before them as uniform scalar loads would be
    const int64_t r_off = offsets[s + (t & 1)];
    const float r_cost = ((t & 2) ? c_w : c_p)[c];
    // the segment's rows: B0 per segment, or those of the table boff
    const long long row0 = boff ? boff[s] : (long long)s * B0;
    const int B = boff ? (int)(boff[s + 1] - row0) : B0;
    const uint32_t *cs = coarse + row0 * kQBuckets;
    const uint32_t *fs = fine + row0 * kQStride;
    {
        const int q = t % kQBuckets, g = t / kQBuckets;
        uint32_t a = 0;
        int bb = g;
        for (; bb + 3 * kG < B; bb += 4 * kG) {
            const uint32_t x0 = cs[(long long)bb * kQBuckets + q];
            const uint32_t x1 = cs[(long long)(bb + kG) * kQBuckets + q];
            const uint32_t x2 = cs[(long long)(bb + 2 * kG) * kQBuckets + q];
            const uint32_t x3 = cs[(long long)(bb + 3 * kG) * kQBuckets + q];
            a += (x0 + x1) + (x2 + x3);
        }
        for (; bb < B; bb += kG) a += cs[(long long)bb * kQBuckets + q];
        part[g][q] = a;
    }
    if (t == 0) sel = -1;
    if (t < 2) s_off[t] = r_off;         // offsets[s], offsets[s + 1]
    if ((t | 2) == 2) s_cost[t >> 1] = r_cost;  // t = 0: c_p[c], t = 2: c_w[c]
    __syncthreads();
    if (t == 0) s_rank = exact_rank(s_cost[0], s_cost[1], s_off[1] - s_off[0]);
    // inclusive scan of the bucket totals (threads 0 .. 255), then the bucket
    // whose range of ranks holds j
    uint32_t tot = 0, incl = 0;
    if (t < kQBuckets) {
#pragma unroll
        for (int g = 0; g < kG; ++g) tot += part[g][t];
        incl = tot;
        for (int d = 1; d < 64; d <<= 1) {
            const uint32_t o = __shfl_up(incl, d, 64);
            if (lane >= d) incl += o;
        }
        if (lane == 63) wsum[wave] = incl;
    }
    __syncthreads();
    const int64_t j = s_rank;
    if (t < kQBuckets) {
        for (int w = 0; w < wave; ++w) incl += wsum[w];
        const int64_t before = (int64_t)(incl - tot);
        if (before < j && j <= (int64_t)incl) {
            sel = t;
            sel_below = before;
        }
    }
    __syncthreads();
    const int bk = sel;  // j is in [1, N] and the totals sum to N, so one bucket holds it
    if (bk < 0) return;
    const int v0 = bk < 128 ? 128 * bk : kQTop / 2 + 128 * (bk - 128);
    {
        // thread t: value v0 + t mod 128 over the rows t / 128, t / 128 + kFG, ...;
        // threads of the first group also count 2^15 in the last bucket
        const int o = t % 128, g = t / 128;
        const int v = v0 + o;
        const int w = v & (kQTop / 2 - 1), sh = (v >> 10) & 16;
        const bool top = bk == kQBuckets - 1 && o == 0;
        uint32_t a = 0, a_top = 0;
        int bb = g;
        for (; bb + 3 * kFG < B; bb += 4 * kFG) {
            const uint32_t x0 = fs[(long long)bb * kQStride + w];
            const uint32_t x1 = fs[(long long)(bb + kFG) * kQStride + w];
            const uint32_t x2 = fs[(long long)(bb + 2 * kFG) * kQStride + w];
            const uint32_t x3 = fs[(long long)(bb + 3 * kFG) * kQStride + w];
            a += ((x0 >> sh) & 0xffffu) + ((x1 >> sh) & 0xffffu) + ((x2 >> sh) & 0xffffu) +
                 ((x3 >> sh) & 0xffffu);
        }
        for (; bb < B; bb += kFG) a += (fs[(long long)bb * kQStride + w] >> sh) & 0xffffu;
        if (top)
            for (int r = g; r < B; r += kFG) a_top += fs[(long long)r * kQStride + kQTop / 2] & 0xffffu;
        fpart[g][o] = a;
        if (o == 0) fpart[g][128] = a_top;
    }
    __syncthreads();
    // scan over the bucket's 129 value slots (threads 0 .. 255; slot 128 is 2^15)
    uint32_t f = 0, fin = 0;
    if (t < kQBuckets) {
        if (t < kF)
#pragma unroll
            for (int g = 0; g < kFG; ++g) f += fpart[g][t];
        fin = f;
        for (int d = 1; d < 64; d <<= 1) {
            const uint32_t o = __shfl_up(fin, d, 64);
            if (lane >= d) fin += o;
        }
        if (lane == 63) wsum[wave] = fin;
    }
    __syncthreads();
    if (t < kF) {
        for (int w = 0; w < wave; ++w) fin += wsum[w];
        const int64_t before = sel_below + (int64_t)(fin - f);
        if (before < j && j <= before + (int64_t)f) q_value[c] = t < 128 ? v0 + t : kQTop;
    }
    if (t == 0) q_rank[c] = j;
}

// classes in a block-uniform loop; the barrier lets the next class reuse the LDS
__global__ __launch_bounds__(kQThreads) void qselect_kernel(const int64_t *offsets,
                                                            const int32_t *seg, const float *c_p,
                                                            const float *c_w, const uint32_t *fine,
                                                            const uint32_t *coarse, int B,
                                                            const int64_t *boff, int C,
                                                            int32_t *q_value, int64_t *q_rank)
{
    for (int c = blockIdx.x; c < C; c += gridDim.x) {
        qselect_class(offsets, seg, c_p, c_w, fine, coarse, B, boff, c, q_value, q_rank);
        __syncthreads();
    }
}

hipError_t select_prepare();
hipError_t qhist_prepare();

hipError_t hist_prepare()
{
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(histogram_kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             (int)(kHistBins * sizeof(uint32_t)));
    if (e != hipSuccess) return e;
    const hipError_t e2 = select_prepare();
    return e2 != hipSuccess ? e2 : qhist_prepare();
}

int hist_parts(int S, long long max_seg, int num_cu)
{
    // about one resident block per compute unit, at least 16K samples per block
    long long B = std::max(1LL, (long long)num_cu / std::max(S, 1));
    B = std::min(B, std::max(1LL, max_seg / 16384));
    return (int)B;
}

hipError_t launch_histogram(const int64_t *offsets, const int32_t *xi, int S, int B,
                            uint32_t *hist, hipStream_t st)
{
    if (S <= 0) return hipSuccess;
    if (B > 1) HIPRET(launch_fill_u32(hist, (long long)S * kHistBins, 0u, st));
    hipLaunchKernelGGL(histogram_kernel, dim3((unsigned)((long long)S * B)), dim3(kHistThreads),
                       kHistBins * sizeof(uint32_t), st, offsets, xi, B, hist);
    return hipGetLastError();
}

// Exact rank j = ceil(c_p N / (c_p + c_w)) in [1, N]: estimate in double,
// then correct with exact 128-bit products.
__device__ int64_t exact_rank(float cp, float cw, int64_t N)
{
    const uint64_t P = (uint64_t)fix33(cp), Wc = (uint64_t)fix33(cw);
    const uint64_t den = P + Wc;
    const unsigned __int128 num = (unsigned __int128)P * (uint64_t)N;
    int64_t j = (int64_t)ceil((double)P / (double)den * (double)N);
    if (j < 1) j = 1;
    if (j > N) j = N;
    while (j > 1 && (unsigned __int128)(uint64_t)(j - 1) * den >= num) --j;
    while (j < N && (unsigned __int128)(uint64_t)j * den < num) ++j;
    return j;
}

// Block per class: prefix counts over the segment histogram; the j-th
// smallest sample is the first value whose cumulative count reaches j.
constexpr int kSelThreads = 1024;

__device__ void select_class(const int64_t *offsets, const int32_t *seg, const float *c_p,
                             const float *c_w, const uint32_t *hist, int c, uint32_t *hl,
                             int32_t *q_value, int64_t *q_rank)
{
    __shared__ uint64_t sc[kSelThreads / 64];
    const int t = threadIdx.x;
    const int s = seg_of_x(seg, c);
    const int64_t N = offsets[s + 1] - offsets[s];
    const uint32_t *h = hist + (long long)s * kHistBins;
    // thread t owns the bins [t * per, (t + 1) * per); per is odd, so a wave's
    // LDS reads fall in distinct banks
    constexpr int per = (kHistBins + kSelThreads - 1) / kSelThreads;
    {   // coalesced loads, all in flight before the first LDS store
        uint32_t r[per];
#pragma unroll
        for (int i = 0; i < per; ++i) {
            const int v = t + i * kSelThreads;
            r[i] = v < kHistBins ? h[v] : 0u;
        }
#pragma unroll
        for (int i = 0; i < per; ++i) {
            const int v = t + i * kSelThreads;
            if (v < kHistBins) hl[v] = r[i];
        }
    }
    const int64_t j = exact_rank(c_p[c], c_w[c], N);
    __syncthreads();
    const int b0 = t * per, b1 = min(kHistBins, b0 + per);
    uint64_t part = 0;
    for (int v = b0; v < b1; ++v) part += hl[v];
    // inclusive scan of the thread totals: within each wave by shuffles, then
    // over the wave totals
    const int lane = t & 63, wave = t >> 6;
    uint64_t incl = part;
    for (int d = 1; d < 64; d <<= 1) {
        const uint64_t o = __shfl_up(incl, d, 64);
        if (lane >= d) incl += o;
    }
    if (lane == 63) sc[wave] = incl;
    __syncthreads();
    if (t == 0)
        for (int w = 1; w < kSelThreads / 64; ++w) sc[w] += sc[w - 1];
    __syncthreads();
    if (wave > 0) incl += sc[wave - 1];
    const uint64_t before = incl - part;
    if ((int64_t)before < j && j <= (int64_t)incl) {
        uint64_t cum = before;
        for (int v = b0; v < b1; ++v) {
            cum += hl[v];
            if ((int64_t)cum >= j) {
                q_value[c] = v;
                break;
            }
        }
    }
    if (t == 0) q_rank[c] = j;
}

// classes in a block-uniform loop; the barrier lets the next class reuse the LDS
__global__ __launch_bounds__(kSelThreads) void select_kernel(const int64_t *offsets,
                                                             const int32_t *seg, const float *c_p,
                                                             const float *c_w, const uint32_t *hist,
                                                             int C, int32_t *q_value, int64_t *q_rank)
{
    extern __shared__ uint32_t hl[];  // the segment's histogram, kHistBins words
    for (int c = blockIdx.x; c < C; c += gridDim.x) {
        select_class(offsets, seg, c_p, c_w, hist, c, hl, q_value, q_rank);
        __syncthreads();
    }
}

hipError_t select_prepare()
{
    return hipFuncSetAttribute(reinterpret_cast<const void *>(select_kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)(kHistBins * sizeof(uint32_t)));
}

hipError_t launch_select(const int64_t *offsets, const int32_t *seg, const float *c_p,
                         const float *c_w, const uint32_t *hist, int C, int32_t *q_value,
                         int64_t *q_rank, hipStream_t st)
{
    hipLaunchKernelGGL(select_kernel, dim3((unsigned)std::min((long long)C, kMaxGridBlocks)),
                       dim3(kSelThreads), kHistBins * sizeof(uint32_t), st, offsets, seg, c_p, c_w,
                       hist, C, q_value, q_rank);
    return hipGetLastError();
}

hipError_t qhist_prepare()
{
    return hipFuncSetAttribute(reinterpret_cast<const void *>(qhist_kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)(2 * kQStride * sizeof(uint32_t)));
}

long long qhist_parts(int S, long long n, int num_cu)
{
    const long long need = (n + kQMaxPart - 1) / kQMaxPart;
    return std::max((long long)hist_parts(S, n, num_cu), std::max(1LL, need));
}

hipError_t launch_class_quantile(const int64_t *offsets, const int32_t *seg, const int32_t *xi,
                                 const float *c_p, const float *c_w, int S, int C, int B,
                                 const int64_t *boff, long long rows, uint32_t *fine,
                                 uint32_t *coarse, int32_t *q_value, int64_t *q_rank,
                                 hipStream_t st)
{
    hipLaunchKernelGGL(qhist_kernel, dim3((unsigned)std::min(rows, kMaxGridBlocks)), dim3(kQThreads),
                       2 * kQStride * sizeof(uint32_t), st, offsets, xi, S, B, boff, rows, fine,
                       coarse);
    HIPRET(hipGetLastError());
    hipLaunchKernelGGL(qselect_kernel, dim3((unsigned)std::min((long long)C, kMaxGridBlocks)),
                       dim3(kQThreads), 0, st, offsets, seg, c_p, c_w, fine, coarse, B, boff, C,
                       q_value, q_rank);
    return hipGetLastError();
}

// ------------------------------------------------------------ block step ----
// Grid indices arriving from the caller (k_prev) are clamped into [0, K).
__device__ __forceinline__ int clampk(int k, int K) { return k < 0 ? 0 : (k >= K ? K - 1 : k); }

// Alg. 1 initialisation r0 = L_in + E[xi]: per class, the exact integer sum of
// the samples (block partial sums added atomically; integer addition makes the
// result independent of the order), then the largest k with eta[k] N <= sum.
__global__ __launch_bounds__(256) void class_sum_kernel(const int64_t *offsets, const int32_t *seg,
                                                        const int32_t *xi, long long chunk,
                                                        unsigned long long *sums)
{
    const int c = blockIdx.x, t = threadIdx.x;
    const int s = seg_of_x(seg, c);
    const long long n0 = offsets[s] + (long long)blockIdx.y * chunk;
    const long long n1 = min(offsets[s + 1], n0 + chunk);
    long long sum = 0;
    for (long long n = n0 + t; n < n1; n += 256) sum += xi[n];
    __shared__ long long sh[256];
    sh[t] = sum;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (t < w) sh[t] += sh[t + w];
        __syncthreads();
    }
    if (t == 0 && sh[0] != 0) atomicAdd(&sums[c], (unsigned long long)sh[0]);
}

__global__ void bcd_init_select_kernel(const int64_t *offsets, const int32_t *seg, const int32_t *eta,
                                       int C, int K, const unsigned long long *sums, int32_t *k0)
{
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    const int s = seg_of_x(seg, c);
    const long long N = offsets[s + 1] - offsets[s];
    const long long tot = (long long)sums[c];
    int lo = 0, hi = K - 1;  // eta ascending: largest k with eta[k] * N <= tot (0 if none)
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if ((long long)eta[mid] * N <= tot) lo = mid;
        else hi = mid - 1;
    }
    k0[c] = lo;
}

hipError_t launch_bcd_init(const int64_t *offsets, const int32_t *seg, const int32_t *xi,
                           const int32_t *eta, int C, int K, long long max_n,
                           unsigned long long *sums, int32_t *k0, hipStream_t st)
{
    const long long chunk = 1 << 16;
    const long long nch = std::max(1LL, (max_n + chunk - 1) / chunk);
    hipLaunchKernelGGL(fill_u32_kernel, dim3((2 * C + 255) / 256), dim3(256), 0, st,
                       reinterpret_cast<uint32_t *>(sums), (long long)2 * C, 0u);
    hipLaunchKernelGGL(class_sum_kernel, dim3(C, (unsigned)nch), dim3(256), 0, st, offsets, seg, xi,
                       chunk, sums);
    hipLaunchKernelGGL(bcd_init_select_kernel, dim3((C + 255) / 256), dim3(256), 0, st, offsets, seg,
                       eta, C, K, (const unsigned long long *)sums, k0);
    return hipGetLastError();
}

// Capacity bound of class c (the memory-capacity constraint of Sec. 3.4), then the largest admissible k.
// The Gauss-Seidel sweep of the block step, one workgroup: for c = 0..C-1 in
// order, thread 0 forms the capacity bound of class c from the other classes'
// current grid points (fp64, no contraction, ascending class order), then the
// block takes the lowest argmin of the exact W[c, 0..kmax_c] (lowest k on
// equal values), which updates k[c] before the next class.  kcur[C] holds the
// state entering the sweep and is updated in place.
constexpr int kSweepThreads = 1024;

__global__ __launch_bounds__(kSweepThreads) void bcd_sweep_kernel(
    const double *W, const int32_t *eta, int C, int K, int G, const float *cap, const float *conc,
    float kappa, int32_t *kcur, int32_t *k_next, double *W_star, uint8_t *feasible,
    double *usage)
{
    __shared__ int s_kmax;
    __shared__ double sw[kSweepThreads / 64];
    __shared__ int sk[kSweepThreads / 64];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const double onek = __dadd_rn(1.0, (double)kappa);
    for (int c = 0; c < C; ++c) {
        if (t == 0) {
            double bound = __builtin_inf();
            for (int g = 0; g < G; ++g) {
                const double u = (double)conc[c * G + g];
                if (!(u > 0.0)) continue;
                double sum = 0.0;
                for (int c2 = 0; c2 < C; ++c2) {
                    if (c2 == c) continue;
                    sum = __dadd_rn(sum, __dmul_rn((double)conc[c2 * G + g],
                                                   (double)eta[clampk(kcur[c2], K)]));
                }
                const double other = __dmul_rn(onek, sum);
                const double b = __ddiv_rn(__dsub_rn((double)cap[g], other), __dmul_rn(onek, u));
                bound = b < bound ? b : bound;
            }
            // eta ascending: the largest k with eta[k] <= bound, or none
            int km = -1, lo = 0, hi = K - 1;
            while (lo <= hi) {
                const int mid = (lo + hi) / 2;
                if ((double)eta[mid] <= bound) {
                    km = mid;
                    lo = mid + 1;
                } else {
                    hi = mid - 1;
                }
            }
            feasible[c] = km >= 0 ? 1 : 0;
            s_kmax = km >= 0 ? km : 0;
        }
        __syncthreads();
        const int kmax = s_kmax;
        const double *w = W + (long long)c * K;
        double bw = __builtin_inf();
        int bk = 0x7fffffff;
        for (int k = t; k <= kmax; k += kSweepThreads)
            if (w[k] < bw) {  // k ascending per thread: its first minimiser
                bw = w[k];
                bk = k;
            }
        for (int d = 32; d > 0; d >>= 1) {
            const double w2 = __shfl_xor(bw, d, 64);
            const int k2 = __shfl_xor(bk, d, 64);
            if (w2 < bw || (w2 == bw && k2 < bk)) {
                bw = w2;
                bk = k2;
            }
        }
        if (lane == 0) {
            sw[wave] = bw;
            sk[wave] = bk;
        }
        __syncthreads();
        if (t == 0) {
            for (int i = 1; i < kSweepThreads / 64; ++i)
                if (sw[i] < bw || (sw[i] == bw && sk[i] < bk)) {
                    bw = sw[i];
                    bk = sk[i];
                }
            kcur[c] = bk;
            W_star[c] = bw;
        }
        __syncthreads();
    }
    for (int g = t; g < G; g += kSweepThreads) {
        double sum = 0.0;
        for (int c = 0; c < C; ++c)
            sum = __dadd_rn(sum, __dmul_rn((double)conc[c * G + g], (double)eta[clampk(kcur[c], K)]));
        usage[g] = __dmul_rn(onek, sum);
    }
    for (int c = t; c < C; c += kSweepThreads) k_next[c] = clampk(kcur[c], K);
}

hipError_t launch_bcd_sweep(const double *W, const int32_t *eta, int C, int K, int G,
                            const float *cap, const float *conc, float kappa, int32_t *kcur,
                            int32_t *k_next, double *W_star, uint8_t *feasible, double *usage,
                            hipStream_t st)
{
    hipLaunchKernelGGL(bcd_sweep_kernel, dim3(1), dim3(kSweepThreads), 0, st, W, eta, C, K, G, cap,
                       conc, kappa, kcur, k_next, W_star, feasible, usage);
    return hipGetLastError();
}

// ------------------------------------------------------------ validation ----
// Block (segment s, part b of B): the smallest and largest sample of its share
// of the segment, merged into mn[s] / mx[s] with atomic min / max (which the
// caller sets to INT_MAX / INT_MIN first); the result does not depend on order.
__global__ __launch_bounds__(256) void seg_minmax_kernel(const int64_t *offsets, const int32_t *xi,
                                                         int B, int32_t *mn, int32_t *mx)
{
    const int s = (int)(blockIdx.x / B), b = (int)(blockIdx.x % B), t = threadIdx.x;
    const long long n0 = offsets[s], N = offsets[s + 1] - n0;
    const long long lo = n0 + (N * b) / B, hi = n0 + (N * (b + 1)) / B;
    int a = 0x7fffffff, c = -0x7fffffff - 1;
    for (long long n = lo + t; n < hi; n += 256) {
        const int v = xi[n];
        a = v < a ? v : a;
        c = v > c ? v : c;
    }
    __shared__ int sa[256], sb[256];
    sa[t] = a;
    sb[t] = c;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (t < w) {
            sa[t] = sa[t + w] < sa[t] ? sa[t + w] : sa[t];
            sb[t] = sb[t + w] > sb[t] ? sb[t + w] : sb[t];
        }
        __syncthreads();
    }
    if (t == 0 && hi > lo) {
        atomicMin(&mn[s], sa[0]);
        atomicMax(&mx[s], sb[0]);
    }
}

hipError_t launch_seg_minmax(const int64_t *offsets, const int32_t *xi, int S, long long max_seg,
                             int32_t *mn, int32_t *mx, hipStream_t st)
{
    // about 16K samples per block, at most 4096 blocks in all
    const long long B = std::max(1LL, std::min(std::max(1LL, 4096LL / S), (max_seg + 16383) / 16384));
    HIPRET(launch_fill_u32(reinterpret_cast<uint32_t *>(mn), S, 0x7fffffffu, st));
    HIPRET(launch_fill_u32(reinterpret_cast<uint32_t *>(mx), S, 0x80000000u, st));
    hipLaunchKernelGGL(seg_minmax_kernel, dim3((unsigned)(S * B)), dim3(256), 0, st, offsets, xi,
                       (int)B, mn, mx);
    return hipGetLastError();
}

}  // namespace dro

namespace dro {

// ============================================================ exact table ====
// The whole table from value counts (the production alternative to the dense
// pass when only results are needed; it does not evaluate per-sample terms).
// For 0 <= x, eta <= L the three candidates of Step 4 reduce to the larger of
// two lines, phi = max(B - a1 x, C - a2 (L - x)) with B = c_w eta,
// C = c_p (L - eta), a1 = min(g, c_w), a2 = min(g, c_p); the first wins exactly
// for (a1 + a2) x <= B - C + a2 L.  With the counts cnt(v) = #{x <= v} and sums
// sum(v) = sum{x : x <= v} of the segment, and t the last sample value on the
// first line's side,
//   S = B cnt(t) - a1 sum(t) + (C - a2 L)(N - cnt(t)) + a2 (sum_all - sum(t)),
// evaluated in 128-bit integers in units of 2^-33: exact.

// Per segment: cnt[v] = #{x <= v} (u32) and sum[v] = sum of the samples <= v
// (u64), from the value histogram, in two passes over blocks of (segment,
// chunk of 4096 bins): the chunk totals, then per chunk the sum of the totals
// before it, the chunk staged in LDS (padded to spread the per-thread runs over
// the banks) and scanned (16 consecutive bins per thread, then across threads),
// and each thread's run of prefixes stored.
constexpr int kPrefixThreads = 256;
constexpr int kPrefixPer = kPrefixChunk / kPrefixThreads;  // 16

__device__ __forceinline__ int pad32(int j) { return j + (j >> 5); }

// Per (segment, chunk): the count and the value-weighted sum of the chunk's
// bins, tot[(s * kPrefixChunks + ch) * 2 + {0, 1}].
__global__ __launch_bounds__(kPrefixThreads) void chunk_total_kernel(const uint32_t *hist,
                                                                     uint64_t *tot)
{
    __shared__ uint64_t rc[kPrefixThreads], rs[kPrefixThreads];
    const int ch = (int)(blockIdx.x % kPrefixChunks), s = (int)(blockIdx.x / kPrefixChunks);
    const int t = threadIdx.x;
    const uint32_t *h = hist + (long long)s * kHistBins;
    const int v0 = ch * kPrefixChunk, v1 = min(kHistBins, v0 + kPrefixChunk);
    uint64_t bc = 0, bs = 0;
    for (int v = v0 + t; v < v1; v += kPrefixThreads) {
        const uint64_t x = h[v];
        bc += x;
        bs += x * (uint64_t)v;
    }
    rc[t] = bc;
    rs[t] = bs;
    __syncthreads();
    for (int w = kPrefixThreads / 2; w > 0; w >>= 1) {
        if (t < w) {
            rc[t] += rc[t + w];
            rs[t] += rs[t + w];
        }
        __syncthreads();
    }
    if (t == 0) {
        tot[(long long)blockIdx.x * 2] = rc[0];
        tot[(long long)blockIdx.x * 2 + 1] = rs[0];
    }
}

__global__ __launch_bounds__(kPrefixThreads) void prefix_kernel(const uint32_t *hist,
                                                                const uint64_t *tot, uint32_t *cnt,
                                                                uint64_t *sum)
{
    __shared__ uint32_t hc[kPrefixChunk + kPrefixChunk / 32];
    __shared__ uint64_t rc[kPrefixThreads / 64], rs[kPrefixThreads / 64];
    const int ch = (int)(blockIdx.x % kPrefixChunks), s = (int)(blockIdx.x / kPrefixChunks);
    const int t = threadIdx.x;
    const uint32_t *h = hist + (long long)s * kHistBins;
    const int v0 = ch * kPrefixChunk, v1 = min(kHistBins, v0 + kPrefixChunk), n = v1 - v0;
    for (int j = t; j < n; j += kPrefixThreads) hc[pad32(j)] = h[v0 + j];
    uint64_t base_c = 0, base_s = 0;  // everything before the chunk, in chunk order
    const uint64_t *tt = tot + (long long)s * kPrefixChunks * 2;
    for (int i = 0; i < ch; ++i) {
        base_c += tt[2 * i];
        base_s += tt[2 * i + 1];
    }
    __syncthreads();
    const int a = t * kPrefixPer;
    uint64_t lc = 0, ls = 0;
    for (int i = 0; i < kPrefixPer; ++i) {
        const int j = a + i;
        if (j < n) {
            const uint64_t x = hc[pad32(j)];
            lc += x;
            ls += x * (uint64_t)(v0 + j);
        }
    }
    // inclusive scans of the thread totals: shuffles within each wave, then
    // the totals of the waves before
    const int lane = t & 63, wave = t >> 6;
    uint64_t ic = lc, is = ls;
    for (int d = 1; d < 64; d <<= 1) {
        const uint64_t oc = __shfl_up(ic, d, 64), os = __shfl_up(is, d, 64);
        if (lane >= d) {
            ic += oc;
            is += os;
        }
    }
    if (lane == 63) {
        rc[wave] = ic;
        rs[wave] = is;
    }
    __syncthreads();
    for (int w = 0; w < wave; ++w) {
        ic += rc[w];
        is += rs[w];
    }
    uint64_t c = base_c + ic - lc, x = base_s + is - ls;
    uint32_t *gc = cnt + (long long)s * kHistBins + v0;
    uint64_t *gs = sum + (long long)s * kHistBins + v0;
    for (int i = 0; i < kPrefixPer; ++i) {
        const int j = a + i;
        if (j < n) {
            const uint64_t hv = hc[pad32(j)];
            c += hv;
            x += hv * (uint64_t)(v0 + j);
            gc[j] = (uint32_t)c;
            gs[j] = x;
        }
    }
}

hipError_t launch_prefix(const uint32_t *hist, int S, uint32_t *cnt, uint64_t *sum, hipStream_t st)
{
    // chunk totals first (after the prefix sums in the same array), then each
    // chunk's scan starts from the totals of the chunks before it
    const long long blocks = (long long)S * kPrefixChunks;
    uint64_t *tot = sum + (long long)S * kHistBins;
    hipLaunchKernelGGL(chunk_total_kernel, dim3((unsigned)blocks), dim3(kPrefixThreads), 0, st,
                       hist, tot);
    hipLaunchKernelGGL(prefix_kernel, dim3((unsigned)blocks), dim3(kPrefixThreads), 0, st, hist,
                       (const uint64_t *)tot, cnt, sum);
    return hipGetLastError();
}

// One wave per (c, k) row, as the minimum over the multipliers of the dense
// path: the wave computes each multiplier's exact S from the segment's prefix
// counts and sums once and stages q_m = RN(S / N) with lambda_m in LDS, a
// chunk of multipliers at a time; then its 64 lanes split into g groups of
// 64/g, g the power of two covering E (at most 64), group j taking radius
// e0 + j and its lanes the multipliers m = part, part + 64/g, ... of the
// chunk.  Each lane keeps the smallest J of its multipliers (the lowest m among
// equal values, as it visits them in ascending order), and log2(64/g) shuffle
// steps take the group's smallest J, ties to the lowest m (W, m_star): the
// same values and the same lowest m as a scan over m.
constexpr int kTableWaves = 4;    // waves (rows) per block
constexpr int kTableChunk = 256;  // multipliers staged per wave at a time

__global__ __launch_bounds__(64 * kTableWaves) void exact_table_kernel(
    const int64_t *offsets, const int32_t *seg, const int32_t *L_, const int32_t *eta_,
    const float *lam, const float *c_p, const float *c_w, const float *eps, const uint32_t *cnt,
    const uint64_t *sum, int E, int C, int K, int M, double *W, int32_t *m_star)
{
    __shared__ double2 stq[kTableWaves][kTableChunk];  // (q_m, lambda_m)
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    // rows in a grid-stride loop of whole waves (no block barrier below)
    for (long long ck = (long long)blockIdx.x * kTableWaves + wv; ck < (long long)C * K;
         ck += (long long)gridDim.x * kTableWaves) {
        const int c = (int)(ck / K), k = (int)(ck % K);
        const int s = seg_of_x(seg, c);
        const int64_t N = offsets[s + 1] - offsets[s];
        const int64_t L = L_[c], eta = eta_[k];
        const uint32_t *cn = cnt + (long long)s * kHistBins;
        const uint64_t *sm = sum + (long long)s * kHistBins;
        const int64_t CP = fix33(c_p[c]), CW = fix33(c_w[c]);
        const double Nd = (double)N;
        int lg = 0;  // log2 of the groups
        while (lg < 6 && (1 << lg) < E) ++lg;
        const int lp = 6 - lg;  // log2 of the lanes per group
        const int part = lane & ((1 << lp) - 1), grp = lane >> lp;
        double2 *q = stq[wv];
        for (int e0 = 0; e0 < E; e0 += 1 << lg) {
            const int e = e0 + grp;
            const double ev = e < E ? (double)eps[(long long)e * C + c] : 0.0;
            double best = __builtin_inf();
            int bm = M;  // no multiplier yet: loses every comparison below
            for (int m0 = 0; m0 < M; m0 += kTableChunk) {
                const int mc = min(kTableChunk, M - m0);
                if (e0 == 0 || M > kTableChunk) {  // else the one chunk is still staged
                    __builtin_amdgcn_wave_barrier();  // the last chunk's reads come first
                    for (int i = lane; i < mc; i += 64) {
                        const float lm = lam[m0 + i];
                        const unsigned __int128 u = exact_S_prefix(cn, sm, N, L, eta, CP, CW, fix33(lm));
                        q[i] = make_double2(__ddiv_rn(fix128_to_double((uint64_t)u, (uint64_t)(u >> 64)), Nd),
                                            (double)lm);
                    }
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
                m_star[o] = bm;
            }
        }
    }
}

// Block per (e, c): lowest k <= kmax with the smallest W, and the values there
// (the exact optimum over a W table whose entries are exact-spec values).
__device__ void table_argmin_row(const double *W, const int32_t *m_star, const int32_t *k_max,
                                int C, int K, int ec, int32_t *k_star, double *W_star,
                                int32_t *m_at_star)
{
    const int c = ec % C, t = threadIdx.x;
    int kmax = K - 1;
    if (k_max) {
        kmax = k_max[c];
        kmax = kmax < 0 ? 0 : (kmax > K - 1 ? K - 1 : kmax);
    }
    const double *w = W + (long long)ec * K;
    double bw = __builtin_inf();
    int bk = 0x7fffffff;
    for (int k = t; k <= kmax; k += 256)
        if (w[k] < bw) {
            bw = w[k];
            bk = k;
        }
    __shared__ double sw[256];
    __shared__ int sk[256];
    sw[t] = bw;
    sk[t] = bk;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (t < s) {
            const double w2 = sw[t + s];
            const int k2 = sk[t + s];
            if (w2 < sw[t] || (w2 == sw[t] && k2 < sk[t])) {
                sw[t] = w2;
                sk[t] = k2;
            }
        }
        __syncthreads();
    }
    if (t == 0) {
        k_star[ec] = sk[0];
        W_star[ec] = sw[0];
        if (m_at_star) m_at_star[ec] = m_star[(long long)ec * K + sk[0]];
    }
}

// rows (e, c) in a block-uniform loop; the barrier lets the next row reuse the LDS
__global__ __launch_bounds__(256) void table_argmin_kernel(const double *W, const int32_t *m_star,
                                                           const int32_t *k_max, int C, int K,
                                                           int rows, int32_t *k_star, double *W_star,
                                                           int32_t *m_at_star)
{
    for (int ec = blockIdx.x; ec < rows; ec += gridDim.x) {
        table_argmin_row(W, m_star, k_max, C, K, ec, k_star, W_star, m_at_star);
        __syncthreads();
    }
}

hipError_t launch_table_argmin(const double *W, const int32_t *m_star, const int32_t *k_max,
                               int E, int C, int K, int32_t *k_star, double *W_star,
                               int32_t *m_at_star, hipStream_t st)
{
    const long long rows = (long long)E * C;  // below 2^31: checked by the entry points
    hipLaunchKernelGGL(table_argmin_kernel, dim3((unsigned)std::min(rows, kMaxGridBlocks)), dim3(256),
                       0, st, W, m_star, k_max, C, K, (int)rows, k_star, W_star, m_at_star);
    return hipGetLastError();
}

hipError_t launch_exact_table(const int64_t *offsets, const int32_t *seg, const int32_t *L,
                              const int32_t *eta, const float *lam, const float *c_p,
                              const float *c_w, const float *eps, const int32_t *k_max,
                              const uint32_t *hist, int S, int E, int C, int K, int M,
                              uint32_t *cnt, uint64_t *sum, double *W, int32_t *m_star,
                              int32_t *k_star, double *W_star, int32_t *m_at_star, hipStream_t st)
{
    HIPRET(launch_prefix(hist, S, cnt, sum, st));
    const long long rows = (long long)C * K;
    const long long blocks = std::min((rows + kTableWaves - 1) / kTableWaves, kMaxGridBlocks);
    hipLaunchKernelGGL(exact_table_kernel, dim3((unsigned)blocks),
                       dim3(64 * kTableWaves), 0, st, offsets, seg, L, eta, lam, c_p, c_w, eps,
                       (const uint32_t *)cnt, (const uint64_t *)sum, E, C, K, M, W, m_star);
    if (k_star) HIPRET(launch_table_argmin(W, m_star, k_max, E, C, K, k_star, W_star, m_at_star, st));
    return hipGetLastError();
}

}  // namespace dro

namespace dro {

// ================================================== baseline reservations ====
// The moment-based and block-aligned baselines of the policy comparison
// (Sec. 5.1: the mean and the block-aligned P95; Sec. 5.4: mean + k sigma), one
// thread per class, exactly in integers:
//   mean_r        = ceil(s / n)
//   lp_r[i]       = min(L, the least integer r with r n - s >= k_i sqrt(n ss - s^2)),
//                   i.e. ceil((s + ceil(sqrt(k_i^2 (n ss - s^2)))) / n)
//   block_r       = q rounded up to a multiple of `block`
// with n, s, ss the count, sum and sum of squares of the class samples.

// ceil(sqrt(d)) for d < 2^100: a double estimate corrected with exact products
__device__ uint64_t ceil_sqrt_u128(unsigned __int128 d)
{
    uint64_t r = (uint64_t)sqrt((double)d);
    while (r > 0 && (unsigned __int128)r * r > d) --r;
    while ((unsigned __int128)(r + 1) * (r + 1) <= d) ++r;
    return r + ((unsigned __int128)r * r < d ? 1u : 0u);
}

__device__ __forceinline__ int64_t ceil_div_pos(__int128 a, int64_t b)
{
    return (int64_t)((a + b - 1) / b);  // a >= 0, b >= 1
}

__global__ void baseline_kernel(int C, const int64_t *count, const int64_t *sum,
                                const int64_t *sumsq, const int32_t *L, BaselineKs ks,
                                const int32_t *q, int block, int32_t *mean_r, int32_t *lp_r,
                                int32_t *block_r)
{
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    const int64_t n = count[c] > 0 ? count[c] : 1, s = sum[c], ss = sumsq[c];
    mean_r[c] = (int32_t)ceil_div_pos(s, n);
    const __int128 v = (__int128)n * ss - (__int128)s * s;  // n^2 times the population variance
    const unsigned __int128 var = v > 0 ? (unsigned __int128)v : 0;
    for (int i = 0; i < ks.n; ++i) {
        const uint64_t k = (uint64_t)ks.k[i];
        const uint64_t r = ceil_sqrt_u128(var * (k * k));
        const int64_t lp = ceil_div_pos((__int128)s + r, n);
        lp_r[(long long)i * C + c] = (int32_t)(lp < L[c] ? lp : L[c]);
    }
    if (q && block_r) {
        const int64_t v0 = q[c] > 0 ? q[c] : 0;
        block_r[c] = (int32_t)(((v0 + block - 1) / block) * block);
    }
}

hipError_t launch_baselines(int C, const int64_t *count, const int64_t *sum, const int64_t *sumsq,
                            const int32_t *L, const BaselineKs &ks, const int32_t *q, int block,
                            int32_t *mean_r, int32_t *lp_r, int32_t *block_r, hipStream_t st)
{
    hipLaunchKernelGGL(baseline_kernel, dim3((C + 255) / 256), dim3(256), 0, st, C, count, sum,
                       sumsq, L, ks, q, block, mean_r, lp_r, block_r);
    return hipGetLastError();
}

// ====================================================== continuous dual ====
// W(eta) = min over gamma >= 0 of gamma eps + S(gamma) / N, the Kantorovich
// dual (Appendix A, Step 3) with gamma continuous (= the LP of Step 5 by
// strong duality).  With a1 = min(g, c_w), a2 = min(g, c_p) the per-sample sup
// is max(B - a1 x, C - a2 (L - x)): convex and piecewise linear in g, so J is
// too, and its right derivative at any g follows from the value counts:
//   dS/dg = -[g < c_w] sum_{x < x0} x - [g < c_p] sum_{x > x0} (L - x)
//           + (#{x = x0}) max(-[g < c_w] x0, -[g < c_p] (L - x0)).
// Bisection on [0, max(c_p, c_w)] (where J' = eps >= 0) finds the smallest g
// with J'(g+) >= 0, i.e. the smallest minimiser; J is evaluated there in fp64.

struct SegStats {
    const uint32_t *cnt;
    const uint64_t *sum;
    double N, SX;
    int tmax;
};

__device__ __forceinline__ void side_stats(const SegStats &g, long long t, double &n, double &s)
{
    if (t < 0) { n = 0.0; s = 0.0; return; }
    if (t > g.tmax) t = g.tmax;
    n = (double)g.cnt[t];
    s = (double)g.sum[t];
}

// value J(g) and right derivative J'(g+) for one (eta, L, costs, eps)
__device__ void dual_at(const SegStats &st, double B, double C, double L, double cw, double cp,
                        double ev, double g, double &J, double &dJ)
{
    const double a1 = g < cw ? g : cw, a2 = g < cp ? g : cp;
    const double s12 = a1 + a2;
    double x0 = s12 > 0.0 ? (B - C + a2 * L) / s12 : (B >= C ? 1e300 : -1e300);
    const double tf = floor(x0 < -2.0 ? -2.0 : (x0 > L + 2.0 ? L + 2.0 : x0));
    const long long t = (long long)tf;
    double n1, s1;  // samples x <= t
    side_stats(st, t, n1, s1);
    // value: line 1 for x <= t, line 2 above (equal at a tie, so ties do not matter)
    const double S = B * n1 - a1 * s1 + (C - a2 * L) * (st.N - n1) + a2 * (st.SX - s1);
    J = g * ev + S / st.N;
    // derivative: ties exactly at x0 take the larger slope
    double nt = 0.0, xt = 0.0;
    if (tf == x0 && t >= 0 && t <= st.tmax) {
        double n0, s0;
        side_stats(st, t - 1, n0, s0);
        nt = n1 - n0;
        xt = (double)t;
        n1 = n0;
        s1 = s0;
    }
    const double w1 = g < cw ? 1.0 : 0.0, w2 = g < cp ? 1.0 : 0.0;
    const double n2 = st.N - n1 - nt, s2 = st.SX - s1 - nt * xt;
    double dS = -w1 * s1 - w2 * (L * n2 - s2);
    if (nt > 0.0) {
        const double d1 = -w1 * xt, d2 = -w2 * (L - xt);
        dS += nt * (d1 > d2 ? d1 : d2);
    }
    dJ = ev + dS / st.N;
}

__global__ __launch_bounds__(256) void continuous_dual_kernel(
    const int64_t *offsets, const int32_t *seg, const int32_t *L_, const int32_t *eta_,
    const float *c_p, const float *c_w, const float *eps, const uint32_t *cnt, const uint64_t *sum,
    int E, int C, int K, double *W, double *gamma)
{
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < (long long)E * C * K;
         i += (long long)gridDim.x * blockDim.x) {
        const int k = (int)(i % K);
        const int ec = (int)(i / K), c = ec % C, e = ec / C;
        const int s = seg_of_x(seg, c);
        SegStats st;
        st.cnt = cnt + (long long)s * kHistBins;
        st.sum = sum + (long long)s * kHistBins;
        st.N = (double)(offsets[s + 1] - offsets[s]);
        st.SX = (double)st.sum[kHistBins - 1];
        const int Li = L_[c];
        st.tmax = Li < kHistBins - 1 ? Li : kHistBins - 1;
        const double L = (double)Li, eta = (double)eta_[k];
        const double cw = (double)c_w[c], cp = (double)c_p[c];
        const double B = cw * eta, Cc = cp * (L - eta);
        const double ev = (double)eps[(long long)e * C + c];
        double J, dJ;
        double lo = 0.0, hi = cw > cp ? cw : cp;
        dual_at(st, B, Cc, L, cw, cp, ev, 0.0, J, dJ);
        if (!(dJ >= 0.0)) {
            for (int it = 0; it < 200 && hi - lo > 0.0; ++it) {
                const double mid = 0.5 * (lo + hi);
                if (mid <= lo || mid >= hi) break;
                dual_at(st, B, Cc, L, cw, cp, ev, mid, J, dJ);
                if (dJ >= 0.0) hi = mid;
                else lo = mid;
            }
            dual_at(st, B, Cc, L, cw, cp, ev, hi, J, dJ);
            lo = hi;
        }
        W[i] = J;
        gamma[i] = lo;
    }
}

hipError_t launch_continuous_dual(const int64_t *offsets, const int32_t *seg, const int32_t *L,
                                  const int32_t *eta, const float *c_p, const float *c_w,
                                  const float *eps, const uint32_t *hist, int S, int E, int C,
                                  int K, uint32_t *cnt, uint64_t *sum, double *W, double *gamma,
                                  hipStream_t st)
{
    HIPRET(launch_prefix(hist, S, cnt, sum, st));
    const long long n = (long long)E * C * K;
    hipLaunchKernelGGL(continuous_dual_kernel, dim3((unsigned)std::min((n + 255) / 256, kMaxGridBlocks)),
                       dim3(256), 0, st,
                       offsets, seg, L, eta, c_p, c_w, eps, (const uint32_t *)cnt,
                       (const uint64_t *)sum, E, C, K, W, gamma);
    return hipGetLastError();
}

}  // namespace dro

namespace dro {

// ===================================================== reservation cost ====
// The stochastic cost of Sec. 3.3, Q(eta, x) = c_p (x - eta)^+ + c_w (eta - x)^+,
// averaged over a class's samples for any given reservations, and the class
// moments from which mean- and spread-based reservations are formed.  Both
// read the value histogram: with cnt(v) = #{x <= v} and sum(v) the sum of
// those samples, for an integer eta
//   sum_n Q(eta, x_n) = c_p ((SX - sum(eta)) - eta (N - cnt(eta)))
//                     + c_w (eta cnt(eta) - sum(eta)),
// evaluated in 128-bit integers in units of 2^-33: exact for every eta.

// One block per class: count, sum, sum of squares and largest sample.
__global__ __launch_bounds__(1024) void moments_kernel(const int32_t *seg, const uint32_t *hist,
                                                       int64_t *count, int64_t *sum,
                                                       int64_t *sumsq, int32_t *xmax)
{
    const int c = blockIdx.x, t = threadIdx.x;
    const uint32_t *h = hist + (long long)seg_of_x(seg, c) * kHistBins;
    unsigned long long n = 0, a = 0, b = 0;
    int mx = -1;
    for (int v = t; v < kHistBins; v += 1024) {
        const unsigned long long k = h[v];
        n += k;
        a += k * (unsigned long long)v;
        b += k * (unsigned long long)v * (unsigned long long)v;
        if (k) mx = v;  // ascending within a thread
    }
    __shared__ unsigned long long sn[1024], sa[1024], sb[1024];
    __shared__ int sm[1024];
    sn[t] = n;
    sa[t] = a;
    sb[t] = b;
    sm[t] = mx;
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
        if (t < w) {
            sn[t] += sn[t + w];
            sa[t] += sa[t + w];
            sb[t] += sb[t + w];
            sm[t] = max(sm[t], sm[t + w]);
        }
        __syncthreads();
    }
    if (t == 0) {
        count[c] = (int64_t)sn[0];
        sum[c] = (int64_t)sa[0];
        sumsq[c] = (int64_t)sb[0];
        xmax[c] = sm[0] < 0 ? 0 : sm[0];
    }
}

// Thread per (row r, class c): cost = RN(RN(S) / N) and cover = cnt(eta).
__global__ __launch_bounds__(256) void reservation_cost_kernel(
    const int64_t *offsets, const int32_t *seg, const float *c_p, const float *c_w,
    const uint32_t *cnt, const uint64_t *sum, int C, long long RC, const int32_t *eta_r,
    double *cost, int64_t *cover)
{
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= RC) return;
    const int c = (int)(i % C);
    const int s = seg_of_x(seg, c);
    const int64_t N = offsets[s + 1] - offsets[s];
    const uint32_t *cn = cnt + (long long)s * kHistBins;
    const uint64_t *sm = sum + (long long)s * kHistBins;
    const __int128 SX = (__int128)sm[kHistBins - 1];
    const int64_t eta = eta_r[i];
    int64_t nle;
    __int128 sle;
    if (eta < 0) {
        nle = 0;
        sle = 0;
    } else if (eta >= kHistBins - 1) {
        nle = N;
        sle = SX;
    } else {
        nle = (int64_t)cn[eta];
        sle = (__int128)sm[eta];
    }
    const __int128 CP = fix33(c_p[c]), CW = fix33(c_w[c]);
    const __int128 S = CP * ((SX - sle) - (__int128)eta * (__int128)(N - nle)) +
                       CW * ((__int128)eta * (__int128)nle - sle);
    const unsigned __int128 u = (unsigned __int128)S;  // S >= 0
    cost[i] = __ddiv_rn(fix128_to_double((uint64_t)u, (uint64_t)(u >> 64)), (double)N);
    cover[i] = nle;
}

hipError_t launch_moments(const int32_t *seg, const uint32_t *hist, int C, int64_t *count,
                          int64_t *sum, int64_t *sumsq, int32_t *xmax, hipStream_t st)
{
    hipLaunchKernelGGL(moments_kernel, dim3(C), dim3(1024), 0, st, seg, hist, count, sum, sumsq,
                       xmax);
    return hipGetLastError();
}

hipError_t launch_reservation_cost(const int64_t *offsets, const int32_t *seg, const float *c_p,
                                   const float *c_w, const uint32_t *hist, int S, int C, int R,
                                   const int32_t *eta_r, uint32_t *cnt, uint64_t *sum,
                                   double *cost, int64_t *cover, hipStream_t st)
{
    HIPRET(launch_prefix(hist, S, cnt, sum, st));
    const long long n = (long long)R * C;
    hipLaunchKernelGGL(reservation_cost_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                       st, offsets, seg, c_p, c_w, (const uint32_t *)cnt, (const uint64_t *)sum,
                       C, n, eta_r, cost, cover);
    return hipGetLastError();
}

}  // namespace dro
