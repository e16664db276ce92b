// C ABI of libdro: argument checks, context and workspace, launch planning.
// Every compute entry point only enqueues work on the caller's stream.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <vector>

#include "dro_internal.h"

struct dro_ctx {
    int device = 0;
    int num_cu = 256;
    int dense_bpc = 1;  // resident dense blocks per compute unit
    void *ws = nullptr;
    size_t ws_size = 0;
    void *scratch = nullptr;    // device address of this device's no-allocation scratch array
    // The host-validated offsets and segment map last staged on the device, and
    // the stream they were staged on: a call whose host arrays and stream match
    // uses the staged copy without uploading it again.
    void *stage = nullptr;
    size_t stage_size = 0;
    bool staged = false;
    hipStream_t staged_stream = nullptr;
    std::vector<int64_t> staged_off;
    std::vector<int32_t> staged_seg;
    char err[1024] = {0};
    // host staging of the configuration-space count table (kept alive until
    // the next configuration search on this context has been enqueued)
    std::vector<long long> ways_h;
    std::vector<int32_t> gpus_h;
    // host copy of the quantile's row table (segments with unequal part counts)
    std::vector<int64_t> qboff_h;
};

// Scratch of dro_cost_eval_noalloc: a fixed array in every device's memory,
// held until the process ends.  Host code never uses its name as an address:
// the device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[DRO_NOALLOC_SCRATCH_BYTES];

namespace {

using namespace dro;

std::mutex g_scratch_mu;
std::vector<void *> g_scratch_ptr;  // indexed by HIP device

// The device address of `scratch` on the current device `dev` (looked up on
// the first call for that device).
hipError_t scratch_address(int dev, void **out)
{
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if ((int)g_scratch_ptr.size() <= dev) g_scratch_ptr.resize(dev + 1, nullptr);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}


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

// Makes ctx's device current for the rest of the calling entry point, or
// returns DRO_EHIP from it when the device cannot be selected.
#define ENTER_DEVICE(ctx)                                                                   \
    DeviceGuard guard_((ctx)->device);                                                      \
    if (!guard_.ok) return fail((ctx), DRO_EHIP, "cannot select device %d", (ctx)->device)

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
    // earlier work may still read the old buffer: on this stream, or on another
    // stream the context was used on before (growth is rare, so wait for all)
    (void)st;
    HIPCHK(hipDeviceSynchronize());
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
    if ((long long)p->K * p->M > 0x7fffffffLL)  // the exact argmin packs (k, m) as k M + m in 31 bits
        return fail(ctx, DRO_ELIMIT, "K*M = %lld exceeds 2^31 - 1 grid pairs", (long long)p->K * p->M);
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

// Tiles of kTM pairs per lane; each tile's samples are split into P slices.
// A problem with at least kDirectSampleTiles (tile, sample) terms per resident
// block runs the persistent grid that claims slices (see dense.hip).  There P
// is the largest of three needs: slices of at most kMaxSliceN samples, so that
// the last ones are short; about kSlicesPerBlock slices per resident block, so
// that the issue priorities keep the blocks of a compute unit in step and the
// blocks still finding work near the end keep every unit full (slices down to
// kBalanceSliceN samples); and one slice for every resident block (slices down
// to kMinSliceN samples).  Measured on 16 x 1e6 samples (K = 2048, M = 256,
// 1024 resident blocks): P = 16 (62,500-sample slices) ran 0.3 % faster than
// the launch of 20,480 short blocks it replaced, P = 31 0.2 % slower and
// P = 8 2.5 % slower.
// A smaller problem (of at most 2^22 blocks) runs one block per slice instead
// (direct mode): a run's set-up (its thresholds, claims, the search for work)
// is then not small beside its work.  P is the smallest whose grid fills its
// last wave of resident blocks to at least 97 %, else the best-filled P
// (P <= 64, slices of at least kMinSliceN samples): on 4 x 1e5 samples
// (K = 512, M = 128) one full wave of blocks (P = 32) ran 3 % faster than two
// (P = 64) and 22 % faster than four.
// The kernels index with the host-validated offsets and segment map: both are
// copied into the workspace at the start of every call, so device data that
// disagrees with the host copies can never steer a kernel outside xi.
constexpr long long kDirectSampleTiles = 65536;
constexpr long long kSlicesPerBlock = 16;
constexpr long long kMaxSliceN = 65536;
constexpr long long kBalanceSliceN = 512;
constexpr long long kMinSliceN = 64;
constexpr long long kMaxDirectSlices = 64;

size_t stage_bytes(const dro_problem *p)
{
    return rup((size_t)(p->S + 1) * 8) + (p->seg_h ? rup((size_t)p->C * 4) : 0);
}

// The offsets (and segment map) every kernel indexes with: the host copies of
// the call, uploaded to the device.  Calls on the workspace keep them in the
// ctx's staging buffer and skip the upload when the host arrays and the stream
// equal the last ones staged; the no-allocation path stages them into its
// arena on every call (the static array is shared by every ctx of the device).
int stage_problem(dro_ctx *ctx, const dro_problem *p, Arena &ar, hipStream_t st, dro_problem *q)
{
    *q = *p;
    const size_t ob = (size_t)(p->S + 1) * 8, sb = p->seg_h ? (size_t)p->C * 4 : 0;
    char *dst;
    if (ar.base != (char *)ctx->ws) {
        dst = ar.take<char>(stage_bytes(p));
    } else {
        const bool same =
            ctx->staged && ctx->staged_stream == st && ctx->staged_off.size() == (size_t)p->S + 1 &&
            std::equal(p->offsets_h, p->offsets_h + p->S + 1, ctx->staged_off.begin()) &&
            (p->seg_h ? ctx->staged_seg.size() == (size_t)p->C &&
                            std::equal(p->seg_h, p->seg_h + p->C, ctx->staged_seg.begin())
                      : ctx->staged_seg.empty());
        if (same) {
            q->offsets = reinterpret_cast<int64_t *>(ctx->stage);
            if (p->seg_h) q->seg = reinterpret_cast<int32_t *>((char *)ctx->stage + rup(ob));
            return DRO_OK;
        }
        ctx->staged = false;
        if (stage_bytes(p) > ctx->stage_size) {
            HIPCHK(hipDeviceSynchronize());  // earlier work may still read the old copy
            if (ctx->stage) HIPCHK(hipFree(ctx->stage));
            ctx->stage = nullptr;
            ctx->stage_size = 0;
            const size_t sz = stage_bytes(p) + (1u << 12);
            if (hipMalloc(&ctx->stage, sz) != hipSuccess) {
                (void)hipGetLastError();
                ctx->stage = nullptr;
                return fail(ctx, DRO_ENOMEM, "staging allocation of %zu bytes failed", sz);
            }
            ctx->stage_size = sz;
        }
        dst = (char *)ctx->stage;
    }
    HIPCHK(hipMemcpyAsync(dst, p->offsets_h, ob, hipMemcpyHostToDevice, st));
    q->offsets = reinterpret_cast<int64_t *>(dst);
    if (p->seg_h) {
        HIPCHK(hipMemcpyAsync(dst + rup(ob), p->seg_h, sb, hipMemcpyHostToDevice, st));
        q->seg = reinterpret_cast<int32_t *>(dst + rup(ob));
    }
    if (dst == (char *)ctx->stage) {
        ctx->staged_off.assign(p->offsets_h, p->offsets_h + p->S + 1);
        if (p->seg_h) ctx->staged_seg.assign(p->seg_h, p->seg_h + p->C);
        else ctx->staged_seg.clear();
        ctx->staged_stream = st;
        ctx->staged = true;
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
    pl.tiles_k = (K + pl.lanes_k - 1) / pl.lanes_k;
    pl.tiles_m = (M + kTM * pl.lanes_m - 1) / (kTM * pl.lanes_m);
    pl.tiles = pl.tiles_k * pl.tiles_m;
    const long long T = (long long)C * pl.tiles;
    const long long slots = (long long)num_cu * std::max(bpc, 1);
    if (T * max_n < kDirectSampleTiles * slots && T * kMaxDirectSlices <= (1LL << 22)) {
        const long long maxP = std::max(1LL, std::min(kMaxDirectSlices, max_n / kMinSliceN));
        long long fillP = 1;
        double best = -1.0;
        for (long long P = 1; P <= maxP; ++P) {
            const long long n = T * P;
            const long long waves = (n + slots - 1) / slots;
            const double fill = (double)n / (double)(waves * slots);
            if (fill > best + 1e-9) {
                best = fill;
                fillP = P;
            }
            if (fill >= 0.97) break;
        }
        pl.P = (int)fillP;
        pl.direct = 1;
        pl.blocks = T * pl.P;
        return pl;
    }
    const long long by_size = (max_n + kMaxSliceN - 1) / kMaxSliceN;
    const long long by_balance = std::min((kSlicesPerBlock * slots + T - 1) / T, max_n / kBalanceSliceN);
    const long long by_fill = std::min((slots + T - 1) / T, max_n / kMinSliceN);
    long long P = std::max({1LL, by_size, by_balance, by_fill});
    P = std::min(P, std::max(1LL, 0x7fffffffLL / T));  // T P claims fit the 32-bit counters
    pl.P = (int)P;
    pl.direct = 0;
    pl.blocks = std::min(slots, T * P);
    return pl;
}

// Claim counters of a dense launch: one per tile and the total.
size_t dense_claim_words(int C, int K, int M)
{
    const DensePlan pl = plan_dense(C, K, M, 1, 1, 1);
    return (size_t)C * pl.tiles + 1;
}

// Host check of the dense entry points, before anything is enqueued: the
// tiles and their claim counters are indexed in 32 bits.
int check_dense(dro_ctx *ctx, const dro_problem *p)
{
    if ((long long)dense_claim_words(p->C, p->K, p->M) > 0x7fffffffLL)
        return fail(ctx, DRO_ELIMIT, "C = %d classes of %zu dense tiles exceed 2^31 - 1 tiles", p->C,
                    dense_claim_words(1, p->K, p->M) - 1);
    return DRO_OK;
}

// Exact S into `S` ([C][K][M] doubles): the dense per-sample sums, then the
// exact epilogue over the segments' prefix counts and sums (cnt, sum).  claim:
// dense_claim_words scratch.
int run_dense(dro_ctx *ctx, const dro_problem *p, double *S, const uint32_t *cnt,
              const uint64_t *sum, const DensePlan &pl, uint32_t *claim, hipStream_t st)
{
    unsigned long long *R = reinterpret_cast<unsigned long long *>(S);
    const long long ckm = (long long)p->C * p->K * p->M;
    const long long T = (long long)p->C * pl.tiles;  // T P < 2^31: check_dense and plan_dense
    HIPCHK(launch_zero_u64_u32(R, ckm, claim, T + 1, st));
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
    a.R = R;
    a.claim = claim;
    HIPCHK(launch_dense(a, st));
    DenseFinishArgs f{};
    f.offsets = p->offsets;
    f.seg = p->seg;
    f.L = p->L;
    f.eta = p->eta;
    f.lam = p->lam;
    f.c_p = p->c_p;
    f.c_w = p->c_w;
    f.cnt = cnt;
    f.sum = sum;
    f.C = p->C;
    f.K = p->K;
    f.M = p->M;
    f.R = R;
    HIPCHK(launch_dense_finish(f, st));
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
    uint32_t *hist;  // [S][kHistBins]
    int B;           // histogram blocks per segment
};

size_t quantile_bytes(const dro_problem *p) { return rup((size_t)p->S * kHistBins * 4); }

QuantBufs take_quantile(Arena &ar, const dro_problem *p, int num_cu)
{
    QuantBufs q;
    q.B = hist_parts(p->S, max_segment(p), num_cu);
    q.hist = ar.take<uint32_t>((size_t)p->S * kHistBins);
    return q;
}

int run_quantile(dro_ctx *ctx, const dro_problem *p, const QuantBufs &qb, int32_t *q_value,
                 int64_t *q_rank, hipStream_t st)
{
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.hist, st));
    HIPCHK(launch_select(p->offsets, p->seg, p->c_p, p->c_w, qb.hist, p->C, q_value, q_rank, st));
    return DRO_OK;
}

// E radius rows of C classes are indexed as e C + c in 32 bits.
int check_rows(dro_ctx *ctx, int E, int C)
{
    if ((long long)E * C > 0x7fffffffLL)
        return fail(ctx, DRO_ELIMIT, "E*C = %lld radius rows exceed 2^31 - 1", (long long)E * C);
    return DRO_OK;
}

bool finite_pos(float v) { return std::isfinite(v) && v > 0.0f; }
bool in_limits(float v) { return v >= 0x1p-10f && v <= 0x1p7f; }

// Scratch of one dense evaluation beyond S: the value histogram, the prefix
// counts and sums, the slice claim counters (and, on the no-allocation path,
// the staged offsets and segment map).
size_t cost_eval_scratch_bytes(const dro_problem *p, bool with_stage)
{
    const size_t bins = (size_t)p->S * kHistBins;
    return (with_stage ? stage_bytes(p) : 0) + quantile_bytes(p) + rup(bins * 4) +
           rup(prefix_sum_words(p->S) * 8) + rup(dense_claim_words(p->C, p->K, p->M) * 4);
}

// The dense evaluation over scratch taken from `ar` (the device must be
// current): value counts and sample sums of every segment, the exact S into
// Sbuf, then the minimum over the multipliers.
int run_cost_eval(dro_ctx *ctx, const dro_problem *p, const Shape &sh, int E, const float *eps,
                  double *W, int32_t *m_star, double *Sbuf, Arena &ar, hipStream_t st)
{
    dro_problem q;
    int rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const DensePlan pl = plan_dense(p->C, p->K, p->M, sh.max_n, ctx->num_cu, ctx->dense_bpc);
    const size_t bins = (size_t)p->S * kHistBins;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    uint32_t *cnt = ar.take<uint32_t>(bins);
    uint64_t *sum = ar.take<uint64_t>(prefix_sum_words(p->S));
    uint32_t *claim = ar.take<uint32_t>(dense_claim_words(p->C, p->K, p->M));
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.hist, st));
    HIPCHK(launch_prefix(qb.hist, p->S, cnt, sum, st));
    rc = run_dense(ctx, p, Sbuf, cnt, sum, pl, claim, st);
    if (rc) return rc;
    HIPCHK(launch_min_over_lambda(Sbuf, p->offsets, p->seg, p->lam, eps, E, p->C, p->K, p->M, W,
                                  m_star, st));
    return DRO_OK;
}

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
    DeviceGuard g(hip_device);
    if (!g.ok) return DRO_EHIP;
    dro_ctx *ctx = new dro_ctx();
    ctx->device = hip_device;
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, hip_device) == hipSuccess && prop.multiProcessorCount > 0)
        ctx->num_cu = prop.multiProcessorCount;
    ctx->dense_bpc = dense_blocks_per_cu();
    if (hist_prepare() != hipSuccess || lp1_prepare() != hipSuccess) {
        (void)hipGetLastError();
        delete ctx;
        return DRO_EHIP;
    }
    // the no-allocation entry point reports DRO_EHIP if this lookup failed
    if (scratch_address(hip_device, &ctx->scratch) != hipSuccess) {
        (void)hipGetLastError();
        ctx->scratch = nullptr;
    }
    *out = ctx;
    return DRO_OK;
}

void dro_destroy(dro_ctx *ctx)
{
    if (!ctx) return;
    DeviceGuard g(ctx->device);  // best effort: destroy returns nothing
    (void)hipDeviceSynchronize();
    if (ctx->ws) (void)hipFree(ctx->ws);
    if (ctx->stage) (void)hipFree(ctx->stage);
    delete ctx;
}

const char *dro_last_error(const dro_ctx *ctx) { return ctx ? ctx->err : "no context"; }

int dro_validate(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                 dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (E < 0 || (E > 0 && !eps)) return fail(ctx, DRO_EINVAL, "bad radius arguments");
    ENTER_DEVICE(ctx);
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
    hipError_t e1 = launch_seg_minmax(p->offsets, p->xi, S, max_segment(p), dmn, dmn + S, st);
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
    if ((rc = check_rows(ctx, E, p->C))) return rc;
    if ((rc = check_dense(ctx, p))) return rc;
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    const size_t ckm = (size_t)p->C * p->K * p->M;
    rc = ensure_ws(ctx, (S ? 0 : rup(ckm * 8)) + cost_eval_scratch_bytes(p, false), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    double *Sbuf = S ? S : ar.take<double>(ckm);
    return run_cost_eval(ctx, p, sh, E, eps, W, m_star, Sbuf, ar, st);
}

int dro_cost_eval_noalloc(dro_ctx *ctx, const dro_problem *p, int32_t E, const float *eps,
                          double *W, int32_t *m_star, double *S, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (E <= 0 || !eps || !W || !S)
        return fail(ctx, DRO_EINVAL, "E must be > 0 and eps, W, S non-NULL");
    if ((rc = check_rows(ctx, E, p->C))) return rc;
    if (!ctx->scratch)
        return fail(ctx, DRO_EHIP, "the scratch array's device address is unknown on device %d",
                    ctx->device);
    const size_t need = cost_eval_scratch_bytes(p, true);
    if (need > (size_t)DRO_NOALLOC_SCRATCH_BYTES)
        return fail(ctx, DRO_ELIMIT,
                    "the problem needs %zu bytes of scratch; the no-allocation array holds %zu",
                    need, (size_t)DRO_NOALLOC_SCRATCH_BYTES);
    if ((rc = check_dense(ctx, p))) return rc;
    ENTER_DEVICE(ctx);
    Arena ar{(char *)ctx->scratch, 0};
    return run_cost_eval(ctx, p, sh, E, eps, W, m_star, S, ar, (hipStream_t)stream);
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
    if ((rc = check_rows(ctx, E, p->C))) return rc;
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    const size_t eck = (size_t)E * p->C * p->K;
    rc = ensure_ws(ctx, rup(eck * 8) + rup(eck * 4), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    double *W = ar.take<double>(eck);
    int32_t *m_star = ar.take<int32_t>(eck);
    // S is exact, so W (the exact-spec J minimised over m) is too, and the
    // lowest-index optimum is a plain minimum over k
    HIPCHK(launch_min_over_lambda(S, p->offsets, p->seg, p->lam, eps, E, p->C, p->K, p->M, W, m_star,
                                  st));
    HIPCHK(launch_table_argmin(W, m_star, k_max, E, p->C, p->K, k_star, W_star, m_at_star, st));
    return DRO_OK;
}

int class_quantile(dro_ctx *ctx, const dro_problem *p, int32_t *q_value, int64_t *q_rank,
                   dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (!q_value || !q_rank) return fail(ctx, DRO_EINVAL, "q_value and q_rank must be non-NULL");
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    // parts per segment (one row of counts each); one count for all segments
    // when they agree, else a row table: segment s owns rows boff[s] .. boff[s+1]
    const int64_t *o = p->offsets_h;
    long long B = 0, rows = 0;
    bool uniform = true;
    for (int s = 0; s < p->S; ++s) {
        const long long b = qhist_parts(p->S, o[s + 1] - o[s], ctx->num_cu);
        if (s == 0) B = b;
        else if (b != B) uniform = false;
        rows += b;
    }
    if (rows > 0x7fffffffLL)
        return fail(ctx, DRO_ELIMIT, "%lld quantile rows exceed 2^31 - 1", rows);
    std::vector<int64_t> &bo = ctx->qboff_h;
    if (!uniform) {
        bo.assign((size_t)p->S + 1, 0);
        for (int s = 0; s < p->S; ++s) bo[s + 1] = bo[s] + qhist_parts(p->S, o[s + 1] - o[s], ctx->num_cu);
    }
    const size_t table = uniform ? 0 : rup(((size_t)p->S + 1) * 8);
    rc = ensure_ws(ctx, rup((size_t)rows * kQStride * 4) + rup((size_t)rows * kQBuckets * 4) + table, st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    uint32_t *fine = ar.take<uint32_t>((size_t)rows * kQStride);
    uint32_t *coarse = ar.take<uint32_t>((size_t)rows * kQBuckets);
    int64_t *boff = nullptr;
    if (!uniform) {  // pageable source: copied out before the call returns
        boff = ar.take<int64_t>((size_t)p->S + 1);
        HIPCHK(hipMemcpyAsync(boff, bo.data(), ((size_t)p->S + 1) * 8, hipMemcpyHostToDevice, st));
    }
    HIPCHK(launch_class_quantile(p->offsets, p->seg, p->xi, p->c_p, p->c_w, p->S, p->C,
                                 uniform ? (int)B : 0, boff, rows, fine, coarse, q_value, q_rank,
                                 st));
    return DRO_OK;
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
    if ((rc = check_rows(ctx, E, p->C))) return rc;
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    const size_t bins = (size_t)p->S * kHistBins;
    rc = ensure_ws(ctx, quantile_bytes(p) + rup(bins * 4) + rup(prefix_sum_words(p->S) * 8), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    uint32_t *cnt = ar.take<uint32_t>(bins);
    uint64_t *sum = ar.take<uint64_t>(prefix_sum_words(p->S));
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.hist, st));
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
    if ((rc = check_rows(ctx, E, p->C))) return rc;
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    const size_t bins = (size_t)p->S * kHistBins;
    rc = ensure_ws(ctx, quantile_bytes(p) + rup(bins * 4) + rup(prefix_sum_words(p->S) * 8), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    uint32_t *cnt = ar.take<uint32_t>(bins);
    uint64_t *sum = ar.take<uint64_t>(prefix_sum_words(p->S));
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.hist, st));
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
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    rc = ensure_ws(ctx, quantile_bytes(p), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.hist, st));
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
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    const size_t bins = (size_t)p->S * kHistBins;
    rc = ensure_ws(ctx, quantile_bytes(p) + rup(bins * 4) + rup(prefix_sum_words(p->S) * 8), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    uint32_t *cnt = ar.take<uint32_t>(bins);
    uint64_t *sum = ar.take<uint64_t>(prefix_sum_words(p->S));
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.hist, st));
    HIPCHK(launch_reservation_cost(p->offsets, p->seg, p->c_p, p->c_w, qb.hist, p->S, p->C, R,
                                   eta_r, cnt, sum, cost, cover, st));
    return DRO_OK;
}

int dro_baseline_reservations(dro_ctx *ctx, int32_t C, const int64_t *count, const int64_t *sum,
                              const int64_t *sumsq, const int32_t *L, int32_t nk,
                              const int32_t *k_sigma_h, const int32_t *q, int32_t block,
                              int32_t *mean_r, int32_t *lp_r, int32_t *block_r,
                              dro_stream_t stream)
{
    if (!ctx) return DRO_EINVAL;
    if (C <= 0 || !count || !sum || !sumsq || !L || !mean_r)
        return fail(ctx, DRO_EINVAL, "C must be > 0 and count, sum, sumsq, L, mean_r non-NULL");
    if (nk < 0 || nk > kMaxBaselineKs || (nk > 0 && (!k_sigma_h || !lp_r)))
        return fail(ctx, DRO_EINVAL, "nk must be in [0, %d], with k_sigma and lp_r when > 0",
                    kMaxBaselineKs);
    if ((q == nullptr) != (block_r == nullptr) || (q && block < 1))
        return fail(ctx, DRO_EINVAL, "q and block_r go together, with block >= 1");
    BaselineKs ks{};
    ks.n = nk;
    for (int i = 0; i < nk; ++i) {
        if (k_sigma_h[i] < 0 || k_sigma_h[i] > 64)
            return fail(ctx, DRO_EINVAL, "k_sigma[%d] = %d outside [0, 64]", i, k_sigma_h[i]);
        ks.k[i] = k_sigma_h[i];
    }
    ENTER_DEVICE(ctx);
    HIPCHK(launch_baselines(C, count, sum, sumsq, L, ks, q, block, mean_r, lp_r, block_r,
                            (hipStream_t)stream));
    return DRO_OK;
}

int bcd_init_state(dro_ctx *ctx, const dro_problem *p, int32_t *k0, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    if (!k0) return fail(ctx, DRO_EINVAL, "k0 must be non-NULL");
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    rc = ensure_ws(ctx, rup((size_t)p->C * 8), st);
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
    if ((rc = check_dense(ctx, p))) return rc;
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    const int C = p->C;
    const DensePlan pl = plan_dense(C, p->K, p->M, sh.max_n, ctx->num_cu, ctx->dense_bpc);
    const size_t ckm = (size_t)C * p->K * p->M;
    const size_t bins = (size_t)p->S * kHistBins;
    const size_t need = rup(ckm * 8) + quantile_bytes(p) + rup(bins * 4) +
                        rup(prefix_sum_words(p->S) * 8) + rup((size_t)C * p->K * 8) +
                        rup((size_t)C * 8) + rup((size_t)C * 4) +
                        rup(dense_claim_words(C, p->K, p->M) * 4);
    rc = ensure_ws(ctx, need, st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    double *S = ar.take<double>(ckm);
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    uint32_t *cnt = ar.take<uint32_t>(bins);
    uint64_t *sum = ar.take<uint64_t>(prefix_sum_words(p->S));
    double *W = ar.take<double>((size_t)C * p->K);
    int64_t *q_rank = ar.take<int64_t>(C);
    int32_t *kcur = ar.take<int32_t>(C);
    uint32_t *claim = ar.take<uint32_t>(dense_claim_words(C, p->K, p->M));

    rc = run_quantile(ctx, p, qb, out->q_value, q_rank, st);
    if (rc) return rc;
    // the quantile's value histogram also gives the prefix counts and sums of
    // the dense epilogue
    HIPCHK(launch_prefix(qb.hist, p->S, cnt, sum, st));
    rc = run_dense(ctx, p, S, cnt, sum, pl, claim, st);
    if (rc) return rc;
    HIPCHK(launch_min_over_lambda(S, p->offsets, p->seg, p->lam, eps, 1, C, p->K, p->M, W, nullptr,
                                  st));
    HIPCHK(hipMemcpyAsync(kcur, k_prev, sizeof(int32_t) * C, hipMemcpyDeviceToDevice, st));
    HIPCHK(launch_bcd_sweep(W, p->eta, C, p->K, grp->G, grp->cap, grp->conc, grp->kappa, kcur,
                            out->k_next, out->W_star, out->feasible, out->usage, st));
    return DRO_OK;
}

}  // extern "C"

// ------------------------------------------------------------------------
// Serving model: routing LP, prefix caching, configuration search, Alg. 1.
// ------------------------------------------------------------------------
namespace {

constexpr int kMaxServiceG = 32;
constexpr long long kMaxConfigs = 1LL << 32;
constexpr double kPiTol = 1e-9;

int check_service(dro_ctx *ctx, int C, const dro_service *v)
{
    if (!ctx) return DRO_EINVAL;
    if (!v) return fail(ctx, DRO_EINVAL, "service is NULL");
    if (C <= 0) return fail(ctx, DRO_EINVAL, "C must be positive (C=%d)", C);
    if (v->G <= 0) return fail(ctx, DRO_EINVAL, "G must be positive (G=%d)", v->G);
    if (v->G > kMaxServiceG)
        return fail(ctx, DRO_ELIMIT, "G=%d exceeds %d configurations", v->G, kMaxServiceG);
    if ((long long)C * v->G > 8192)
        return fail(ctx, DRO_ELIMIT, "C*G=%lld exceeds 8192 routing variables", (long long)C * v->G);
    if (!v->tau || !v->pp || !v->tau_h || !v->pp_h || !v->Mcap || !v->Cc || !v->Bc || !v->lam ||
        !v->Lin || !v->Lpre || !v->D)
        return fail(ctx, DRO_EINVAL, "a required array of the service model is NULL");
    if (v->J <= 0 || v->J > 4096) return fail(ctx, DRO_ELIMIT, "J=%d outside [1, 4096]", v->J);
    const float sc[] = {v->alpha, v->beta, v->t_ar, v->c_gpu, v->c_slo, v->c_rej, v->kappa};
    for (float x : sc)
        if (!std::isfinite(x) || x < 0.0f)
            return fail(ctx, DRO_EINVAL, "service constants must be finite and >= 0");
    if (!(v->u_max > 0.0f && v->u_max < 1.0f))
        return fail(ctx, DRO_EINVAL, "u_max=%g must lie in (0, 1)", (double)v->u_max);
    if (v->NL < 0) return fail(ctx, DRO_EINVAL, "NL must be >= 0");
    for (int g = 0; g < v->G; ++g)
        if (v->tau_h[g] < 1 || v->pp_h[g] < 1 || (long long)v->tau_h[g] * v->pp_h[g] > 4096)
            return fail(ctx, DRO_EINVAL, "configuration %d: tau=%d pp=%d", g, v->tau_h[g], v->pp_h[g]);
    return DRO_OK;
}

SvcArgs svc_args(const dro_service *v, int C)
{
    SvcArgs s;
    s.C = C;
    s.G = v->G;
    s.tau = v->tau;
    s.pp = v->pp;
    s.Mcap = v->Mcap;
    s.Cc = v->Cc;
    s.Bc = v->Bc;
    s.lam = v->lam;
    s.Lin = v->Lin;
    s.Lpre = v->Lpre;
    s.D = v->D;
    s.alpha = v->alpha;
    s.beta = v->beta;
    s.t_ar = v->t_ar;
    s.NL = (double)v->NL;
    s.c_gpu = v->c_gpu;
    s.c_slo = v->c_slo;
    s.c_rej = v->c_rej;
    s.kappa = v->kappa;
    s.u_max = v->u_max;
    s.J = v->J;
    return s;
}

// ways[g][b] = number of (z_g, .., z_{G-1}) >= 0 with sum z_h gpus_h <= b,
// saturating; fills ctx->ways_h and ctx->gpus_h and returns |Z| (or -1).
long long count_configs(dro_ctx *ctx, const dro_service *v, hipStream_t st)
{
    // an earlier search may still be copying the previous table
    if (!ctx->ways_h.empty() && hipStreamSynchronize(st) != hipSuccess) return -1;
    const int G = v->G, J = v->J;
    ctx->gpus_h.assign(G, 0);
    for (int g = 0; g < G; ++g) ctx->gpus_h[g] = v->tau_h[g] * v->pp_h[g];
    std::vector<long long> &w = ctx->ways_h;
    w.assign((size_t)(G + 1) * (J + 1), 0);
    const long long cap = 1LL << 62;
    for (int b = 0; b <= J; ++b) w[(size_t)G * (J + 1) + b] = 1;
    for (int g = G - 1; g >= 0; --g)
        for (int b = 0; b <= J; ++b) {
            long long acc = 0;
            for (int u = 0; u * ctx->gpus_h[g] <= b; ++u) {
                acc += w[(size_t)(g + 1) * (J + 1) + (b - u * ctx->gpus_h[g])];
                if (acc > cap) acc = cap;
            }
            w[(size_t)g * (J + 1) + b] = acc;
        }
    return w[J];
}

size_t config_bytes(int C, int G, int J, long long nz)
{
    const long long nb = (nz + 255) / 256;
    return rup(config_pre_doubles(C, G) * 8) + rup((size_t)G * 4) + rup((size_t)(G + 1) * (J + 1) * 8) +
           rup((size_t)G * 4) + rup((size_t)nb * 8) * 3 + 3 * rup(8) + rup(4 * 8);
}

struct ConfigBufs {
    double *pre_d;
    int32_t *route, *gpus;
    long long *ways;
    double *part_obj;
    long long *part_rank, *part_feas;
    double *best_obj;
    long long *best_rank, *n_feas;
    int32_t *flag;
};

ConfigBufs take_config(Arena &ar, int C, int G, int J, long long nz)
{
    const long long nb = (nz + 255) / 256;
    ConfigBufs b;
    b.pre_d = ar.take<double>(config_pre_doubles(C, G));
    b.route = ar.take<int32_t>(G);
    b.ways = ar.take<long long>((size_t)(G + 1) * (J + 1));
    b.gpus = ar.take<int32_t>(G);
    b.part_obj = ar.take<double>(nb);
    b.part_rank = ar.take<long long>(nb);
    b.part_feas = ar.take<long long>(nb);
    b.best_obj = ar.take<double>(1);
    b.best_rank = ar.take<long long>(1);
    b.n_feas = ar.take<long long>(1);
    b.flag = ar.take<int32_t>(8);
    return b;
}

int upload_configs(dro_ctx *ctx, const ConfigBufs &b, int G, int J, hipStream_t st)
{
    HIPCHK(hipMemcpyAsync(b.ways, ctx->ways_h.data(), sizeof(long long) * (size_t)(G + 1) * (J + 1),
                          hipMemcpyHostToDevice, st));
    HIPCHK(hipMemcpyAsync(b.gpus, ctx->gpus_h.data(), sizeof(int32_t) * G, hipMemcpyHostToDevice, st));
    return DRO_OK;
}

int max_pivots(int C, int G) { return 50 * (3 * C + G + C * G) + 1000; }

}  // namespace

extern "C" {

int bcd_service_times(dro_ctx *ctx, const dro_problem *p, const dro_service *svc, double *T,
                      double *ET2, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    rc = check_service(ctx, p->C, svc);
    if (rc) return rc;
    if (!T || !ET2) return fail(ctx, DRO_EINVAL, "T and ET2 must be non-NULL");
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    const int C = p->C;
    rc = ensure_ws(ctx, quantile_bytes(p) + 4 * rup((size_t)C * 8), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    int64_t *cnt = ar.take<int64_t>(C), *sum = ar.take<int64_t>(C), *ssq = ar.take<int64_t>(C);
    int32_t *xmax = ar.take<int32_t>(C);
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.hist, st));
    HIPCHK(launch_moments(p->seg, qb.hist, C, cnt, sum, ssq, xmax, st));
    HIPCHK(launch_service_times(svc_args(svc, C), cnt, sum, ssq, T, ET2, st));
    return DRO_OK;
}

int bcd_queue_state(dro_ctx *ctx, int32_t C, const dro_service *svc, const double *T,
                    const double *ET2, const double *pi, const int32_t *z, const int32_t *eta_c,
                    const uint8_t *delta, double *Wq, double *cap, double *conc, double *mem,
                    dro_stream_t stream)
{
    int rc = check_service(ctx, C, svc);
    if (rc) return rc;
    if (!T || !ET2 || !pi || !z || !eta_c || !delta || !Wq || !cap || !conc)
        return fail(ctx, DRO_EINVAL, "a queue-state argument is NULL");
    ENTER_DEVICE(ctx);
    HIPCHK(launch_state(svc_args(svc, C), T, ET2, pi, z, eta_c, delta, Wq, cap, conc, mem,
                        (hipStream_t)stream));
    return DRO_OK;
}

int bcd_routing_lp(dro_ctx *ctx, int32_t C, const dro_service *svc, const double *Wc,
                   const double *T, const double *Wq, const int32_t *z, const int32_t *eta_c,
                   const uint8_t *delta, double *pi, double *lp_objective, int32_t *info,
                   dro_stream_t stream)
{
    int rc = check_service(ctx, C, svc);
    if (rc) return rc;
    if (!Wc || !T || !Wq || !z || !eta_c || !delta || !pi || !lp_objective || !info)
        return fail(ctx, DRO_EINVAL, "a routing-LP argument is NULL");
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    const int G = svc->G, m = 2 * C + G;
    rc = ensure_ws(ctx, rup(lp1_tableau_doubles(C, G) * 8) + rup((size_t)m * 4), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    double *work = ar.take<double>(lp1_tableau_doubles(C, G));
    int32_t *basis = ar.take<int32_t>(m);
    HIPCHK(launch_lp1(svc_args(svc, C), Wc, T, Wq, z, eta_c, delta, work, basis, max_pivots(C, G),
                      pi, lp_objective, info, st));
    return DRO_OK;
}

int bcd_reservation_sweep(dro_ctx *ctx, int32_t C, int32_t K, const double *W,
                          const int32_t *eta, int32_t G, const double *conc, const double *cap,
                          float kappa, const int32_t *k_in, int32_t *k_out, uint8_t *feasible,
                          dro_stream_t stream)
{
    if (!ctx) return DRO_EINVAL;
    if (C <= 0 || K <= 0 || G <= 0 || !W || !eta || !conc || !cap || !k_in || !k_out)
        return fail(ctx, DRO_EINVAL, "sweep needs C, K, G > 0 and non-NULL W, eta, conc, cap, k");
    if (!std::isfinite(kappa) || kappa < 0.0f) return fail(ctx, DRO_EINVAL, "kappa must be >= 0");
    if (k_in == k_out) return fail(ctx, DRO_EINVAL, "k_in and k_out must differ");
    ENTER_DEVICE(ctx);
    HIPCHK(launch_sweep(W, eta, C, K, G, conc, cap, kappa, k_in, k_out, feasible,
                        (hipStream_t)stream));
    return DRO_OK;
}

int bcd_prefix_cache(dro_ctx *ctx, int32_t C, int32_t G, const double *conc, uint8_t *delta,
                     dro_stream_t stream)
{
    if (!ctx) return DRO_EINVAL;
    if (C <= 0 || G <= 0 || !conc || !delta)
        return fail(ctx, DRO_EINVAL, "prefix cache needs C, G > 0 and non-NULL conc, delta");
    ENTER_DEVICE(ctx);
    HIPCHK(launch_cache(conc, C * G, delta, (hipStream_t)stream));
    return DRO_OK;
}

int bcd_config_search(dro_ctx *ctx, int32_t C, const dro_service *svc, const double *Wc,
                      const double *T, const double *ET2, const double *pi,
                      const int32_t *eta_c, const uint8_t *delta, int32_t *z,
                      double *best_objective, int64_t *best_rank, int64_t *n_feasible,
                      dro_stream_t stream)
{
    int rc = check_service(ctx, C, svc);
    if (rc) return rc;
    if (!Wc || !T || !ET2 || !pi || !eta_c || !delta || !z)
        return fail(ctx, DRO_EINVAL, "a configuration-search argument is NULL");
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    const long long nz = count_configs(ctx, svc, st);
    if (nz < 0) return fail(ctx, DRO_EHIP, "stream synchronisation failed");
    if (nz > kMaxConfigs)
        return fail(ctx, DRO_ELIMIT, "%lld configurations exceed 2^32", nz);
    const int G = svc->G, J = svc->J;
    rc = ensure_ws(ctx, config_bytes(C, G, J, nz), st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    const ConfigBufs b = take_config(ar, C, G, J, nz);
    rc = upload_configs(ctx, b, G, J, st);
    if (rc) return rc;
    HIPCHK(launch_config_search(svc_args(svc, C), nz, b.gpus, b.ways, Wc, T, ET2, pi, eta_c, delta,
                                b.pre_d, b.route, b.part_obj, b.part_rank, b.part_feas, z, nullptr,
                                nullptr, best_objective ? best_objective : b.best_obj,
                                best_rank ? (long long *)best_rank : b.best_rank,
                                n_feasible ? (long long *)n_feasible : b.n_feas, b.flag, st));
    return DRO_OK;
}

int dro_bcd_solve(dro_ctx *ctx, const dro_problem *p, const float *eps, const dro_service *svc,
                  int32_t max_outer, int32_t max_inner, int32_t *z, int32_t *k, double *pi,
                  uint8_t *delta, double *objective, int32_t *info, dro_stream_t stream)
{
    Shape sh;
    int rc = check_problem(ctx, p, &sh);
    if (rc) return rc;
    rc = check_service(ctx, p->C, svc);
    if (rc) return rc;
    if (!eps || !z || !k || !pi || !delta || !objective || !info)
        return fail(ctx, DRO_EINVAL, "a solver argument is NULL");
    if (max_outer <= 0 || max_inner <= 0)
        return fail(ctx, DRO_EINVAL, "max_outer and max_inner must be positive");
    ENTER_DEVICE(ctx);
    hipStream_t st = (hipStream_t)stream;
    const int C = p->C, G = svc->G, K = p->K, J = svc->J, CG = C * G, m = 2 * C + G;
    const long long nz = count_configs(ctx, svc, st);
    if (nz < 0) return fail(ctx, DRO_EHIP, "stream synchronisation failed");
    if (nz > kMaxConfigs) return fail(ctx, DRO_ELIMIT, "%lld configurations exceed 2^32", nz);
    const size_t bins = (size_t)p->S * kHistBins;
    const size_t need = quantile_bytes(p) + rup(bins * 4) +
                        rup(prefix_sum_words(p->S) * 8) + rup((size_t)C * K * 8) + rup((size_t)C * K * 4) +
                        4 * rup((size_t)C * 8) + rup(lp1_tableau_doubles(C, G) * 8) +
                        rup((size_t)m * 4) + 4 * rup((size_t)CG * 8) + 2 * rup((size_t)CG) +
                        7 * rup((size_t)G * 8) + 6 * rup((size_t)C * 8) +
                        config_bytes(C, G, J, nz) + rup(64);
    rc = ensure_ws(ctx, need, st);
    if (rc) return rc;
    Arena ar{(char *)ctx->ws, 0};
    dro_problem q;
    rc = stage_problem(ctx, p, ar, st, &q);
    if (rc) return rc;
    p = &q;
    const SvcArgs s = svc_args(svc, C);
    const QuantBufs qb = take_quantile(ar, p, ctx->num_cu);
    uint32_t *pcnt = ar.take<uint32_t>(bins);
    uint64_t *psum = ar.take<uint64_t>(prefix_sum_words(p->S));
    double *W = ar.take<double>((size_t)C * K);
    int32_t *mstar = ar.take<int32_t>((size_t)C * K);
    int64_t *cnt = ar.take<int64_t>(C), *sum = ar.take<int64_t>(C), *ssq = ar.take<int64_t>(C);
    int32_t *xmax = ar.take<int32_t>(C);
    double *work = ar.take<double>(lp1_tableau_doubles(C, G));
    int32_t *basis = ar.take<int32_t>(m);
    double *T = ar.take<double>(CG), *ET2 = ar.take<double>(CG), *pi_new = ar.take<double>(CG);
    double *conc = ar.take<double>(CG);
    uint8_t *d_new = ar.take<uint8_t>(CG), *feas = ar.take<uint8_t>(C);
    double *Wq = ar.take<double>(G), *cap = ar.take<double>(G), *lpobj = ar.take<double>(1);
    double *Wq_blk = ar.take<double>(G);
    double *Wc = ar.take<double>(C);
    int32_t *eta_c = ar.take<int32_t>(C), *k_new = ar.take<int32_t>(C);
    unsigned long long *sums = ar.take<unsigned long long>(C);
    int32_t *ctl = ar.take<int32_t>(8);  // converge flag, lp pivots, lp status
    const ConfigBufs cb = take_config(ar, C, G, J, nz);
    rc = upload_configs(ctx, cb, G, J, st);
    if (rc) return rc;

    // the exact worst-case table of the radius row, the moments, the service times, r0
    HIPCHK(launch_histogram(p->offsets, p->xi, p->S, qb.B, qb.hist, st));
    HIPCHK(launch_exact_table(p->offsets, p->seg, p->L, p->eta, p->lam, p->c_p, p->c_w, eps, nullptr,
                              qb.hist, p->S, 1, C, K, p->M, pcnt, psum, W, mstar, nullptr, nullptr,
                              nullptr, st));
    HIPCHK(launch_moments(p->seg, qb.hist, C, cnt, sum, ssq, xmax, st));
    HIPCHK(launch_service_times(s, cnt, sum, ssq, T, ET2, st));
    HIPCHK(launch_bcd_init(p->offsets, p->seg, p->xi, p->eta, C, K, sh.max_n, sums, k, st));
    HIPCHK(launch_fill_u32(reinterpret_cast<uint32_t *>(pi), 2LL * CG, 0u, st));
    HIPCHK(launch_zero_u8(delta, CG, st));

    int outer = 0, inner = 0, pivots = 0, status = 0;
    const int mp = max_pivots(C, G);
    for (int it = 0; it < max_outer; ++it) {
        ++outer;
        bool converged = false;
        // the wait is linearised once per Block 1, at the state entering it
        HIPCHK(launch_gather(W, p->eta, k, C, K, Wc, eta_c, st));
        HIPCHK(launch_state(s, T, ET2, pi, z, eta_c, delta, Wq_blk, cap, conc, nullptr, st));
        for (int jt = 0; jt < max_inner; ++jt) {
            ++inner;
            HIPCHK(launch_gather(W, p->eta, k, C, K, Wc, eta_c, st));
            HIPCHK(launch_lp1(s, Wc, T, Wq_blk, z, eta_c, delta, work, basis, mp, pi_new, lpobj,
                              ctl + 1, st));
            HIPCHK(launch_state(s, T, ET2, pi_new, z, eta_c, delta, Wq, cap, conc, nullptr, st));
            HIPCHK(launch_sweep(W, p->eta, C, K, G, conc, cap, svc->kappa, k, k_new, feas, st));
            HIPCHK(launch_converge(C, G, kPiTol, k_new, k, pi_new, pi, ctl, st));
            int32_t h[3];
            HIPCHK(hipMemcpyAsync(h, ctl, sizeof(h), hipMemcpyDeviceToHost, st));
            HIPCHK(hipStreamSynchronize(st));
            pivots += h[1];
            if (h[2] == 1) status |= 1;
            if (h[2] == 2) status |= 2;
            if (h[2] == 3) status |= 4;
            if (h[0]) {
                converged = true;
                break;
            }
        }
        if (!converged) status |= 16;
        // Block 2, then Block 3 with the new delta
        HIPCHK(launch_gather(W, p->eta, k, C, K, Wc, eta_c, st));
        HIPCHK(launch_state(s, T, ET2, pi, z, eta_c, delta, Wq, cap, conc, nullptr, st));
        HIPCHK(launch_cache(conc, CG, d_new, st));
        HIPCHK(launch_config_search(s, nz, cb.gpus, cb.ways, Wc, T, ET2, pi, eta_c, d_new, cb.pre_d,
                                    cb.route, cb.part_obj, cb.part_rank, cb.part_feas, z, d_new,
                                    delta, cb.best_obj, cb.best_rank, cb.n_feas, cb.flag, st));
        int32_t changed = 0;
        HIPCHK(hipMemcpyAsync(&changed, cb.flag, sizeof(changed), hipMemcpyDeviceToHost, st));
        HIPCHK(hipStreamSynchronize(st));
        if (!changed) break;
        if (it == max_outer - 1) status |= 32;
    }
    HIPCHK(launch_gather(W, p->eta, k, C, K, Wc, eta_c, st));
    HIPCHK(launch_state_objective(s, T, ET2, pi, z, eta_c, delta, Wc, cb.pre_d, cb.route,
                                  objective, st));
    std::vector<uint8_t> fh(C);
    HIPCHK(hipMemcpyAsync(fh.data(), feas, C, hipMemcpyDeviceToHost, st));
    HIPCHK(hipStreamSynchronize(st));
    for (int c = 0; c < C; ++c)
        if (!fh[c]) status |= 8;
    info[0] = outer;
    info[1] = inner;
    info[2] = pivots;
    info[3] = status;
    return DRO_OK;
}

}  // extern "C"
