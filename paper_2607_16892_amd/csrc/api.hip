// C ABI of libdro: argument checks, context and workspace, launch planning.
// Every compute entry point only enqueues work on the caller's stream.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <vector>

#include "dro_internal.h"

struct dro_ctx {
    int device = 0;
    int num_cu = 256;
    int dense_bpc = 1;  // resident dense blocks per compute unit
    void *ws = nullptr;
    size_t ws_size = 0;
    uint32_t *flags = nullptr;  // device word of DRO_FLAG_* bits
    char err[1024] = {0};
};

namespace {

using namespace dro;

int fail(dro_ctx *ctx, int code, const char *fmt, ...)
{
    if (ctx) {
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(ctx->err, sizeof(ctx->err), fmt, ap);
        va_end(ap);
    }
    return code;
}

#define HIPCHK(expr)                                                                       \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess)                                                              \
            return fail(ctx, DRO_EHIP, "%s: %s", #expr, hipGetErrorString(e_));           \
    } while (0)

// Makes the context's device current for the duration of a call.
struct DeviceGuard {
    int prev = -1;
    bool ok = true;
    explicit DeviceGuard(int dev)
    {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard()
    {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

// Bump allocator over the context workspace.
struct Arena {
    char *base = nullptr;
    size_t off = 0;
    template <class T> T *take(size_t count)
    {
        off = (off + 255) & ~size_t(255);
        T *p = reinterpret_cast<T *>(base + off);
        off += count * sizeof(T);
        return p;
    }
};

size_t rup(size_t v) { return (v + 255) & ~size_t(255); }

int ensure_ws(dro_ctx *ctx, size_t need, hipStream_t st)
{
    if (need <= ctx->ws_size) return DRO_OK;
    // earlier work on this stream may still read the old buffer
    HIPCHK(hipStreamSynchronize(st));
    if (ctx->ws) {
        HIPCHK(hipFree(ctx->ws));
        ctx->ws = nullptr;
        ctx->ws_size = 0;
    }
    const size_t sz = need + need / 4 + (1u << 20);
    if (hipMalloc(&ctx->ws, sz) != hipSuccess) {
        (void)hipGetLastError();
        ctx->ws = nullptr;
        return fail(ctx, DRO_ENOMEM, "workspace allocation of %zu bytes failed", sz);
    }
    ctx->ws_size = sz;
    return DRO_OK;
}

struct Shape {
    long long max_n = 0;  // largest class sample count
};

// Host-visible checks shared by every entry point.
int check_problem(dro_ctx *ctx, const dro_problem *p, Shape *sh)
{
    if (!ctx) return DRO_EINVAL;
    if (!p) return fail(ctx, DRO_EINVAL, "problem is NULL");
    if (p->C <= 0 || p->S <= 0 || p->K <= 0 || p->M <= 0)
        return fail(ctx, DRO_EINVAL, "C, S, K and M must be positive (C=%d S=%d K=%d M=%d)", p->C,
                    p->S, p->K, p->M);
    if (!p->offsets || !p->offsets_h || !p->xi || !p->L || !p->eta || !p->lam || !p->c_p || !p->c_w)
        return fail(ctx, DRO_EINVAL, "a required array of the problem is NULL");
    if ((p->seg == nullptr) != (p->seg_h == nullptr))
        return fail(ctx, DRO_EINVAL, "seg and seg_h must both be given or both be NULL");
    if (!p->seg && p->S != p->C)
        return fail(ctx, DRO_EINVAL, "without a segment map S must equal C (S=%d C=%d)", p->S, p->C);
    if (p->K > 32769) return fail(ctx, DRO_ELIMIT, "K=%d exceeds 2^15 + 1 grid points", p->K);
    if (p->M > 65536) return fail(ctx, DRO_ELIMIT, "M=%d exceeds 65536 multipliers", p->M);
    const int64_t *o = p->offsets_h;
    if (o[0] != 0) return fail(ctx, DRO_EINVAL, "offsets[0] must be 0");
    for (int s = 0; s < p->S; ++s)
        if (o[s + 1] < o[s]) return fail(ctx, DRO_EINVAL, "offsets decrease at segment %d", s);
    long long mx = 0;
    for (int c = 0; c < p->C; ++c) {
        const int s = p->seg_h ? p->seg_h[c] : c;
        if (s < 0 || s >= p->S)
            return fail(ctx, DRO_EINVAL, "seg[%d] = %d outside [0, %d)", c, s, p->S);
        const long long n = o[s + 1] - o[s];
        if (n <= 0) return fail(ctx, DRO_EINVAL, "class %d has an empty sample segment", c);
        if (n > (1LL << 26))
            return fail(ctx, DRO_ELIMIT, "class %d has %lld samples (> 2^26)", c, n);
        mx = std::max(mx, n);
    }
    sh->max_n = mx;
    return DRO_OK;
}

// Tiles of kTK x kTM pairs per lane; samples of a class split into P slices so
// that the grid fills whole waves of resident blocks (cap = CUs x blocks/CU):
// the smallest P whose last wave is at least 97 % full, slices >= 1024 samples.
// The kernels index with the host-validated offsets and segment map: both are
// copied into the workspace at the start of every call, so device data that
// disagrees with the host copies can never steer a kernel outside xi.
size_t stage_bytes(const dro_problem *p)
{
    return rup((size_t)(p->S + 1) * 8) + (p->seg_h ? rup((size_t)p->C * 4) : 0);
}

int stage_problem(dro_ctx *ctx, const dro_problem *p, Arena &ar, hipStream_t st, dro_problem *q)
{
    *q = *p;
    int64_t *off = ar.take<int64_t>((size_t)p->S + 1);
    HIPCHK(hipMemcpyAsync(off, p->offsets_h, (size_t)(p->S + 1) * 8, hipMemcpyHostToDevice, st));
    q->offsets = off;
    if (p->seg_h) {
        int32_t *seg = ar.take<int32_t>((size_t)p->C);
        HIPCHK(hipMemcpyAsync(seg, p->seg_h, (size_t)p->C * 4, hipMemcpyHostToDevice, st));
        q->seg = seg;
    }
    return DRO_OK;
}

DensePlan plan_dense(int C, int K, int M, long long max_n, int num_cu, int bpc)
{
    DensePlan pl{};
    const int need_m = (M + kTM - 1) / kTM;
    pl.lanes_m = 1;
    while (pl.lanes_m < need_m && pl.lanes_m < kThreads) pl.lanes_m *= 2;
    pl.lanes_k = kThreads / pl.lanes_m;
    pl.tiles_k = (K + kTK * pl.lanes_k - 1) / (kTK * pl.lanes_k);
    pl.tiles_m = (M + kTM * pl.lanes_m - 1) / (kTM * pl.lanes_m);
    const long long base = (long long)C * pl.tiles_k * pl.tiles_m;
    const long long cap = (long long)num_cu * std::max(bpc, 1);
    const long long maxP = std::max(1LL, std::min(64LL, max_n / 1024));
    long long bestP = 1;
    double best = -1.0;
    for (long long P = 1; P <= maxP; ++P) {
        const long long n = base * P;
        const long long waves = (n + cap - 1) / cap;
        const double fill = (double)n / (double)(waves * cap);
        if (fill > best + 1e-9) {
            best = fill;
            bestP = P;
        }
        if (fill >= 0.97) break;
    }
    pl.P = (int)bestP;
    pl.blocks = base * bestP;
    return pl;
}

int refine_slices(long long max_n) { return (int)std::min(256LL, std::max(1LL, max_n / 8192)); }

// S (approximate) into `S`, using `part` when the plan splits samples.
int run_dense(dro_ctx *ctx, const dro_problem *p, const Shape &sh, double *S, double *part,
              const DensePlan &pl, hipStream_t st)
{
    DenseArgs a{};
    a.offsets = p->offsets;
    a.seg = p->seg;
    a.xi = p->xi;
    a.L = p->L;
    a.eta = p->eta;
    a.lam = p->lam;
    a.c_p = p->c_p;
    a.c_w = p->c_w;
    a.C = p->C;
    a.K = p->K;
    a.M = p->M;
    a.plan = pl;
    a.out = pl.P > 1 ? part : S;
    HIPCHK(launch_dense(a, st));
    if (pl.P > 1) HIPCHK(launch_reduce_slices(part, pl.P, (long long)p->C * p->K * p->M, S, st));
    (void)sh;
    return DRO_OK;
}

size_t dense_bytes(const dro_problem *p, const DensePlan &pl, bool need_S)
{
    const size_t ckm = (size_t)p->C * p->K * p->M;
    size_t b = 0;
    if (need_S) b += rup(ckm * sizeof(double));
    if (pl.P > 1) b += rup((size_t)pl.P * ckm * sizeof(double));
    return b;
}

struct RefineBufs {
    int32_t *cand, *count;
    double *thresh, *chunk_min;
    uint64_t *part;
};

size_t band_chunks(int K) { return (size_t)(K + kBandKC - 1) / kBandKC; }

size_t refine_bytes(int EC, int P, int K)
{
    return rup((size_t)EC * kBandCap * 4) + rup((size_t)EC * 4) + rup((size_t)EC * 8) +
           rup((size_t)EC * band_chunks(K) * 8) + rup((size_t)EC * kBandCap * P * 16);
}

RefineBufs take_refine(Arena &ar, int EC, int P, int K)
{
    RefineBufs r;
    r.cand = ar.take<int32_t>((size_t)EC * kBandCap);
    r.count = ar.take<int32_t>(EC);
    r.thresh = ar.take<double>(EC);
    r.chunk_min = ar.take<double>((size_t)EC * band_chunks(K));
    r.part = ar.take<uint64_t>((size_t)EC * kBandCap * P * 2);
    return r;
}

// Screen, refine and finalize for all (e, c) (c_only < 0) or for one class.
int run_argmin(dro_ctx *ctx, const dro_problem *p, int E, const float *eps, const double *S,
               const int32_t *k_max, int e_row, int c_only, const RefineBufs &rb, int P,
               int32_t *k_star, double *W_star, int32_t *m_at_star, hipStream_t st)
{
    const int EC = E * p->C;
    BandArgs b{};
    b.S = S;
    b.offsets = p->offsets;
    b.seg = p->seg;
    b.L = p->L;
    b.lam = p->lam;
    b.c_p = p->c_p;
    b.c_w = p->c_w;
    b.eps = eps;
    b.k_max = k_max;
    b.E = E;
    b.C = p->C;
    b.K = p->K;
    b.M = p->M;
    b.e_row = e_row;
    b.c_only = c_only;
    b.cand = rb.cand;
    b.count = rb.count;
    b.thresh = rb.thresh;
    b.flags = ctx->flags;
    HIPCHK(launch_band(b, rb.chunk_min, st));

    RefineArgs r{};
    r.offsets = p->offsets;
    r.seg = p->seg;
    r.xi = p->xi;
    r.L = p->L;
    r.eta = p->eta;
    r.lam = p->lam;
    r.c_p = p->c_p;
    r.c_w = p->c_w;
    r.cand = rb.cand;
    r.count = rb.count;
    r.C = p->C;
    r.M = p->M;
    r.EC = EC;
    r.P = P;
    r.e_row = e_row;
    r.c_only = c_only;
    r.part = rb.part;
    HIPCHK(launch_refine(r, st));

    FinalArgs f{};
    f.offsets = p->offsets;
    f.seg = p->seg;
    f.lam = p->lam;
    f.eps = eps;
    f.cand = rb.cand;
    f.count = rb.count;
    f.thresh = rb.thresh;
    f.part = rb.part;
    f.C = p->C;
    f.M = p->M;
    f.EC = EC;
    f.P = P;
    f.e_row = e_row;
    f.c_only = c_only;
    f.k_star = k_star;
    f.W_star = W_star;
    f.m_at_star = m_at_star;
    f.flags = ctx->flags;
    HIPCHK(launch_finalize(f, st));
    return DRO_OK;
}

long long max_segment(const dro_problem *p)
{
    long long max_seg = 0;
    for (int s = 0; s < p->S; ++s)
        max_seg = std::max(max_seg, (long long)(p->offsets_h[s + 1] - p->offsets_h[s]));
    return max_seg;
}

struct QuantBufs {
    uint32_t *hist, *part;
    int B;
};

size_t quantile_bytes(const dro_problem *p, int num_cu)
{
    const int B = hist_parts(p->S, max_segment(p), num_cu);
    return rup((size_t)p->S * kHistBins * 4) + (B > 1 ? rup((size_t)p->S * B * kHistBins * 4) : 0);
}

QuantBufs take_quantile(Arena &ar, const dro_problem *p, int num_cu)
{
    QuantBufs q;
    q.B = hist_parts(p->S, max_segment(p), num_cu);
    q.hist = ar.take<uint32_t>((size_t)p->S * kHistBins);
    q.part = q.B > 1 ? ar.take<uint32_t>((size_t)p->S * q.B * kHistBins) : nullptr;
    return q;
}

int run_quantile(dro_ctx *ctx, const dro_problem *p, const QuantBufs &qb, int32_t *q_value,
                 int64_t *q_rank, hipStream_t st)
{
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.part, qb.hist, st));
    HIPCHK(launch_select(p->offsets, p->seg, p->c_p, p->c_w, qb.hist, p->C, q_value, q_rank, st));
    return DRO_OK;
}

bool finite_pos(float v) { return std::isfinite(v) && v > 0.0f; }
bool in_limits(float v) { return v >= 0x1p-10f && v <= 0x1p7f; }

}  // namespace

// ============================================================== C ABI ====

extern "C" {

const char *dro_strerror(int code)
{
    switch (code) {
    case DRO_OK: return "ok";
    case DRO_EINVAL: return "invalid argument";
    case DRO_ERANGE: return "device data out of range";
    case DRO_ENOMEM: return "out of device memory";
    case DRO_EHIP: return "HIP runtime error";
    case DRO_ELIMIT: return "beyond the exactness limits";
    default: return "unknown error";
    }
}

int dro_create(int hip_device, dro_ctx **out)
{
    if (!out) return DRO_EINVAL;
    *out = nullptr;
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || hip_device < 0 || hip_device >= n)
        return DRO_EINVAL;
    dro_ctx *ctx = new dro_ctx();
    ctx->device = hip_device;
    DeviceGuard g(hip_device);
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, hip_device) == hipSuccess && prop.multiProcessorCount > 0)
        ctx->num_cu = prop.multiProcessorCount;
    ctx->dense_bpc = dense_blocks_per_cu();
    if (hist_prepare() != hipSuccess) {
        (void)hipGetLastError();
        delete ctx;
        return DRO_EHIP;
    }
    if (hipMalloc(&ctx->flags, sizeof(uint32_t)) != hipSuccess ||
        hipMemset(ctx->flags, 0, sizeof(uint32_t)) != hipSuccess) {
        delete ctx;
        return DRO_ENOMEM;
    }
    *out = ctx;
    return DRO_OK;
}

void dro_destroy(dro_ctx *ctx)
{
    if (!ctx) return;
    DeviceGuard g(ctx->device);
    (void)hipDeviceSynchronize();
    if (ctx->ws) (void)hipFree(ctx->ws);
    if (ctx->flags) (void)hipFree(ctx->flags);
    delete ctx;
}

const char *dro_last_error(const dro_ctx *ctx) { return ctx ? ctx->err : "no context"; }

int dro_take_flags(dro_ctx *ctx, uint32_t *flags_out)
{
    if (!ctx || !flags_out) return fail(ctx, DRO_EINVAL, "NULL argument");
    DeviceGuard g(ctx->device);
    HIPCHK(hipDeviceSynchronize());
    HIPCHK(hipMemcpy(flags_out, ctx->flags, sizeof(uint32_t), hipMemcpyDeviceToHost));
    HIPCHK(hipMemset(ctx->flags, 0, sizeof(uint32_t)));
    return DRO_OK;
}

int dro_validate(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                 dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (E < 0 || (E > 0 && !eps)) return fail(ctx, DRO_EINVAL, "bad radius arguments");
    DeviceGuard g(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    const int C = p->C, S = p->S, K = p->K, M = p->M;
    std::vector<int64_t> off(S + 1);
    std::vector<int32_t> seg(C), L(C), eta(K), mn(S), mx(S);
    std::vector<float> lam(M), cp(C), cw(C), ev((size_t)E * C);
    HIPCHK(hipStreamSynchronize(st));
    HIPCHK(hipMemcpy(off.data(), p->offsets, (S + 1) * 8, hipMemcpyDeviceToHost));
    if (p->seg) HIPCHK(hipMemcpy(seg.data(), p->seg, C * 4, hipMemcpyDeviceToHost));
    else for (int c = 0; c < C; ++c) seg[c] = c;
    HIPCHK(hipMemcpy(L.data(), p->L, C * 4, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(eta.data(), p->eta, K * 4, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(lam.data(), p->lam, M * 4, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(cp.data(), p->c_p, C * 4, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(cw.data(), p->c_w, C * 4, hipMemcpyDeviceToHost));
    if (E > 0) HIPCHK(hipMemcpy(ev.data(), eps, (size_t)E * C * 4, hipMemcpyDeviceToHost));
    for (int s = 0; s <= S; ++s)
        if (off[s] != p->offsets_h[s])
            return fail(ctx, DRO_ERANGE, "device offsets[%d] = %lld differ from the host copy %lld",
                        s, (long long)off[s], (long long)p->offsets_h[s]);
    for (int c = 0; c < C; ++c)
        if (seg[c] != (p->seg_h ? p->seg_h[c] : c))
            return fail(ctx, DRO_ERANGE, "device seg[%d] differs from the host copy", c);
    int32_t minL = 1 << 30;
    for (int c = 0; c < C; ++c) {
        if (L[c] < 0) return fail(ctx, DRO_ERANGE, "L[%d] = %d is negative", c, L[c]);
        if (L[c] > (1 << 15)) return fail(ctx, DRO_ELIMIT, "L[%d] = %d exceeds 2^15", c, L[c]);
        minL = std::min(minL, L[c]);
    }
    for (int k = 0; k < K; ++k) {
        if (eta[k] < 0 || eta[k] > minL)
            return fail(ctx, DRO_ERANGE, "eta[%d] = %d outside [0, min L = %d]", k, eta[k], minL);
        if (k && eta[k] <= eta[k - 1])
            return fail(ctx, DRO_ERANGE, "eta is not strictly ascending at %d", k);
    }
    for (int m = 0; m < M; ++m) {
        if (!finite_pos(lam[m])) return fail(ctx, DRO_ERANGE, "lam[%d] is not finite and > 0", m);
        if (m && !(lam[m] > lam[m - 1]))
            return fail(ctx, DRO_ERANGE, "lam is not strictly ascending at %d", m);
        if (!in_limits(lam[m]))
            return fail(ctx, DRO_ELIMIT, "lam[%d] = %g outside [2^-10, 2^7]", m, (double)lam[m]);
    }
    for (int c = 0; c < C; ++c) {
        if (!finite_pos(cp[c]) || !finite_pos(cw[c]))
            return fail(ctx, DRO_ERANGE, "c_p/c_w of class %d not finite and > 0", c);
        if (!in_limits(cp[c]) || !in_limits(cw[c]))
            return fail(ctx, DRO_ELIMIT, "c_p/c_w of class %d outside [2^-10, 2^7]", c);
    }
    for (size_t i = 0; i < ev.size(); ++i)
        if (!std::isfinite(ev[i]) || ev[i] < 0.0f)
            return fail(ctx, DRO_ERANGE, "eps[%zu] is negative or not finite", i);
    // min / max of every segment on the device
    int32_t *dmn = nullptr;
    HIPCHK(hipMalloc(&dmn, sizeof(int32_t) * 2 * S));
    hipError_t e1 = launch_seg_minmax(p->offsets, p->xi, S, dmn, dmn + S, st);
    hipError_t e2 = e1 == hipSuccess ? hipStreamSynchronize(st) : e1;
    hipError_t e3 = e2 == hipSuccess ? hipMemcpy(mn.data(), dmn, 4 * S, hipMemcpyDeviceToHost) : e2;
    hipError_t e4 = e3 == hipSuccess ? hipMemcpy(mx.data(), dmn + S, 4 * S, hipMemcpyDeviceToHost) : e3;
    (void)hipFree(dmn);
    HIPCHK(e4);
    for (int c = 0; c < C; ++c) {
        const int s = seg[c];
        if (off[s + 1] == off[s]) continue;
        if (mn[s] < 0 || mx[s] > L[c])
            return fail(ctx, DRO_ERANGE, "class %d has samples outside [0, L=%d] (min %d, max %d)",
                        c, L[c], mn[s], mx[s]);
    }
    return DRO_OK;
}

int dro_cost_eval(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps, double *W,
                  int32_t *m_star, double *S, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (E <= 0 || !eps || !W) return fail(ctx, DRO_EINVAL, "E must be > 0 and eps, W non-NULL");
    DeviceGuard g(ctx->device);
    if (!g.ok) return fail(ctx, DRO_EHIP, "cannot select device %d", ctx->device);
    hipStream_t st = (hipStream_t)stream;
    const DensePlan pl = plan_dense(p->C, p->K, p->M, sh.max_n, ctx->num_cu, ctx->dense_bpc);
    rc = ensure_ws(ctx, stage_bytes(p) + dense_bytes(p, pl, S == nullptr), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const size_t ckm = (size_t)p->C * p->K * p->M;
    double *Sbuf = S ? S : ar.take<double>(ckm);
    double *part = pl.P > 1 ? ar.take<double>((size_t)pl.P * ckm) : nullptr;
    rc = run_dense(ctx, p, sh, Sbuf, part, pl, st);
    if (rc) return rc;
    HIPCHK(launch_min_over_lambda(Sbuf, p->offsets, p->seg, p->lam, eps, E, p->C, p->K, p->M, W,
                                  m_star, st));
    return DRO_OK;
}

int dro_argmin_reservation(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                           const double *S, const int32_t *k_max, int32_t *k_star, double *W_star,
                           int32_t *m_at_star, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (E <= 0 || !eps || !S || !k_star || !W_star)
        return fail(ctx, DRO_EINVAL, "E must be > 0 and eps, S, k_star, W_star non-NULL");
    DeviceGuard g(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    const int EC = E * p->C;
    const int P = refine_slices(sh.max_n);
    rc = ensure_ws(ctx, stage_bytes(p) + refine_bytes(EC, P, p->K), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    RefineBufs rb = take_refine(ar, EC, P, p->K);
    return run_argmin(ctx, p, E, eps, S, k_max, 0, -1, rb, P, k_star, W_star, m_at_star, st);
}

int class_quantile(dro_ctx *ctx, const dro_problem *p, int32_t *q_value, int64_t *q_rank,
                   dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (!q_value || !q_rank) return fail(ctx, DRO_EINVAL, "q_value and q_rank must be non-NULL");
    DeviceGuard g(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    rc = ensure_ws(ctx, stage_bytes(p) + quantile_bytes(p, ctx->num_cu), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    return run_quantile(ctx, p, qb, q_value, q_rank, st);
}

int dro_exact_table(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                    const int32_t *k_max, double *W, int32_t *m_star, int32_t *k_star,
                    double *W_star, int32_t *m_at_star, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (E <= 0 || !eps || !W || !m_star || (k_star && !W_star))
        return fail(ctx, DRO_EINVAL, "E must be > 0 and eps, W, m_star (and W_star with k_star) non-NULL");
    DeviceGuard g(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    const size_t bins = (size_t)p->S * kHistBins;
    rc = ensure_ws(ctx, stage_bytes(p) + quantile_bytes(p, ctx->num_cu) + rup(bins * 4) + rup(bins * 8), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    uint32_t *cnt = ar.take<uint32_t>(bins);
    uint64_t *sum = ar.take<uint64_t>(bins);
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.part, qb.hist, st));
    HIPCHK(launch_exact_table(p->offsets, p->seg, p->L, p->eta, p->lam, p->c_p, p->c_w, eps, k_max,
                              qb.hist, p->S, E, p->C, p->K, p->M, cnt, sum, W, m_star, k_star,
                              W_star, m_at_star, st));
    return DRO_OK;
}

int dro_continuous_dual(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                        double *W, double *gamma, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (E <= 0 || !eps || !W || !gamma)
        return fail(ctx, DRO_EINVAL, "E must be > 0 and eps, W, gamma non-NULL");
    DeviceGuard g(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    const size_t bins = (size_t)p->S * kHistBins;
    rc = ensure_ws(ctx, stage_bytes(p) + quantile_bytes(p, ctx->num_cu) + rup(bins * 4) + rup(bins * 8), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    uint32_t *cnt = ar.take<uint32_t>(bins);
    uint64_t *sum = ar.take<uint64_t>(bins);
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.part, qb.hist, st));
    HIPCHK(launch_continuous_dual(p->offsets, p->seg, p->L, p->eta, p->c_p, p->c_w, eps, qb.hist,
                                  p->S, E, p->C, p->K, cnt, sum, W, gamma, st));
    return DRO_OK;
}

int class_moments(dro_ctx *ctx, const dro_problem *p, int64_t *count, int64_t *sum,
                  int64_t *sumsq, int32_t *xmax, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (!count || !sum || !sumsq || !xmax)
        return fail(ctx, DRO_EINVAL, "count, sum, sumsq and xmax must be non-NULL");
    DeviceGuard g(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    rc = ensure_ws(ctx, stage_bytes(p) + quantile_bytes(p, ctx->num_cu), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.part, qb.hist, st));
    HIPCHK(launch_moments(p->seg, qb.hist, p->C, count, sum, sumsq, xmax, st));
    return DRO_OK;
}

int dro_reservation_cost(dro_ctx *ctx, const dro_problem *p, int32_t R, const int32_t *eta_r,
                         double *cost, int64_t *cover, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (R <= 0 || !eta_r || !cost || !cover)
        return fail(ctx, DRO_EINVAL, "R must be > 0 and eta_r, cost, cover non-NULL");
    if ((long long)R * p->C > (1LL << 31))
        return fail(ctx, DRO_ELIMIT, "R*C = %lld reservations exceed 2^31", (long long)R * p->C);
    DeviceGuard g(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    const size_t bins = (size_t)p->S * kHistBins;
    rc = ensure_ws(ctx, stage_bytes(p) + quantile_bytes(p, ctx->num_cu) + rup(bins * 4) + rup(bins * 8), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    uint32_t *cnt = ar.take<uint32_t>(bins);
    uint64_t *sum = ar.take<uint64_t>(bins);
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.part, qb.hist, st));
    HIPCHK(launch_reservation_cost(p->offsets, p->seg, p->c_p, p->c_w, qb.hist, p->S, p->C, R,
                                   eta_r, cnt, sum, cost, cover, st));
    return DRO_OK;
}

int bcd_init_state(dro_ctx *ctx, const dro_problem *p, int32_t *k0, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (!k0) return fail(ctx, DRO_EINVAL, "k0 must be non-NULL");
    DeviceGuard g(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    rc = ensure_ws(ctx, stage_bytes(p) + rup((size_t)p->C * 8), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    unsigned long long *sums = ar.take<unsigned long long>(p->C);
    HIPCHK(launch_bcd_init(p->offsets, p->seg, p->xi, p->eta, p->C, p->K, sh.max_n, sums, k0, st));
    return DRO_OK;
}

int bcd_block_step(dro_ctx *ctx, const dro_problem *p, const float *eps, const dro_groups *grp,
                   const int32_t *k_prev, dro_step_out *out, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (!eps || !grp || !k_prev || !out || !out->k_next || !out->W_star || !out->q_value ||
        !out->usage || !out->feasible)
        return fail(ctx, DRO_EINVAL, "a block-step argument or output is NULL");
    if (grp->G <= 0 || !grp->cap || !grp->conc || !std::isfinite(grp->kappa) || grp->kappa < 0.0f)
        return fail(ctx, DRO_EINVAL, "groups need G > 0, cap, conc and a finite kappa >= 0");
    DeviceGuard g(ctx->device);
    hipStream_t st = (hipStream_t)stream;
    const int C = p->C;
    const DensePlan pl = plan_dense(C, p->K, p->M, sh.max_n, ctx->num_cu, ctx->dense_bpc);
    const int P = refine_slices(sh.max_n);
    const size_t need = dense_bytes(p, pl, true) + quantile_bytes(p, ctx->num_cu) +
                        refine_bytes(C, P, p->K) + rup((size_t)C * 8) + 3 * rup((size_t)C * 4);
    rc = ensure_ws(ctx, stage_bytes(p) + need, st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const size_t ckm = (size_t)C * p->K * p->M;
    double *S = ar.take<double>(ckm);
    double *part = pl.P > 1 ? ar.take<double>((size_t)pl.P * ckm) : nullptr;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    RefineBufs rb = take_refine(ar, C, P, p->K);
    int64_t *q_rank = ar.take<int64_t>(C);
    int32_t *kmax = ar.take<int32_t>(C);
    int32_t *kcur = ar.take<int32_t>(C);

    rc = run_quantile(ctx, p, qb, out->q_value, q_rank, st);
    if (rc) return rc;
    rc = run_dense(ctx, p, sh, S, part, pl, st);
    if (rc) return rc;
    HIPCHK(hipMemcpyAsync(kcur, k_prev, sizeof(int32_t) * C, hipMemcpyDeviceToDevice, st));
    for (int c = 0; c < C; ++c) {
        HIPCHK(launch_bcd_kmax(p->eta, C, p->K, grp->G, grp->cap, grp->conc, grp->kappa, kcur, c,
                               kmax, out->feasible, st));
        rc = run_argmin(ctx, p, 1, eps, S, kmax, 0, c, rb, P, kcur, out->W_star, nullptr, st);
        if (rc) return rc;
    }
    HIPCHK(launch_bcd_finish(p->eta, C, p->K, grp->G, grp->conc, grp->kappa, kcur, out->usage,
                             out->k_next, st));
    return DRO_OK;
}

}  // extern "C"
