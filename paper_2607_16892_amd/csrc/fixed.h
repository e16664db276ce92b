// Fixed-point helpers shared by the dense and exact translation units.
//
// Inside the library's limits (integers <= 2^15, binary32 coefficients in
// [2^-10, 2^7]) every candidate of phi (Appendix A, Step 4) is an integer
// multiple of 2^-33 below 2^56.  The helpers below form those integers, divide
// them exactly, and round 128-bit sums of them to double once.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dro {

// v * 2^33 for a binary32 v in [2^-10, 2^7] (exact integer below 2^41).
__device__ __forceinline__ int64_t fix33(float v)
{
    const uint32_t bits = __float_as_uint(v);
    const int e = (int)((bits >> 23) & 0xffu);
    const int64_t mant = (int64_t)((bits & 0x7fffffu) | 0x800000u);
    const int sh = e - 117;  // e - 127 - 23 + 33
    return sh >= 0 ? (mant << sh) : (mant >> (-sh));
}

// floor(a / b) for b > 0 and |a| < 2^62: a double estimate corrected with
// exact integer products, so the result does not depend on the estimate.
__device__ __forceinline__ int64_t floor_div(int64_t a, int64_t b)
{
    int64_t q = (int64_t)floor((double)a / (double)b);
    while (q * b > a) --q;
    while ((q + 1) * b <= a) ++q;
    return q;
}

// Correctly rounded double of the unsigned 128-bit value (hi, lo) times 2^-33.
__device__ inline double fix128_to_double(uint64_t lo, uint64_t hi)
{
    int nb;
    if (hi) nb = 128 - __clzll((long long)hi);
    else if (lo) nb = 64 - __clzll((long long)lo);
    else return 0.0;
    if (nb <= 53) return ldexp((double)(long long)lo, -33);
    const int sh = nb - 53;
    const unsigned __int128 v = ((unsigned __int128)hi << 64) | (unsigned __int128)lo;
    uint64_t mant = (uint64_t)(v >> sh);
    const unsigned __int128 rem = v & ((((unsigned __int128)1) << sh) - 1);
    const unsigned __int128 half = ((unsigned __int128)1) << (sh - 1);
    if (rem > half || (rem == half && (mant & 1u))) mant += 1;
    return ldexp((double)(long long)mant, sh - 33);
}

// Correctly rounded double of a signed 128-bit value times 2^-33.
__device__ inline double sfix128_to_double(__int128 v)
{
    const bool neg = v < 0;
    const unsigned __int128 u = neg ? (unsigned __int128)(-v) : (unsigned __int128)v;
    const double d = fix128_to_double((uint64_t)u, (uint64_t)(u >> 64));
    return neg ? -d : d;
}

// The two lines of phi for one (class, grid point, multiplier), in units of
// 2^-33.  For 0 <= x, eta <= L the three candidates of Step 4 reduce to the
// larger of  B - A1 x  and  Cc - A2 (L - x)  with B = c_w eta, Cc = c_p (L - eta),
// A1 = min(g, c_w), A2 = min(g, c_p) (Q(eta, x) is itself the larger of
// c_w (eta - x) and c_p (x - eta), and for x, L - x >= 0 the smaller slope wins
// each pair).  Their difference is  y2 - y1 = De x - Nu  with De = A1 + A2 and
// Nu = B - Cc + A2 L, so the lines cross at x0 = Nu / De.
struct PairLinesFix {
    int64_t B, Cc, A1, A2, Nu, De;
};

__device__ __forceinline__ PairLinesFix pair_lines_fix(int64_t CP, int64_t CW, int64_t G,
                                                       int64_t eta, int64_t L)
{
    PairLinesFix q;
    q.B = CW * eta;
    q.Cc = CP * (L - eta);
    q.A1 = G < CW ? G : CW;
    q.A2 = G < CP ? G : CP;
    q.De = q.A1 + q.A2;
    q.Nu = q.B - q.Cc + q.A2 * L;
    return q;
}

}  // namespace dro
