"""class_quantile against the oracle's order statistic, on the cases that stress
its layout: 16-bit counts packed two to a word (values below and above 2^14),
the value 2^15 itself, ranks on the first and last value of a coarse bucket,
segments long enough to need more blocks than the default, segments with
unequal block counts (many short segments beside one long one, read through
a row table), classes aliasing one segment, constant samples, and cost ratios
that put the rank at 1 or N
(Prop. 4.2: the critical fractile c_p / (c_p + c_w), read as the
generalised-inverse order statistic).  Bar: q_value and q_rank bit for bit.
"""
import numpy as np
import pytest

import oracle
from workloads.configs import Workload, _csr, _f32, eta_grid, lam_grid

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ctx(dev):
    import paper_2607_16892_amd as dro
    c = dro.Context(dev.index or 0)
    yield c
    c.close()


def _workload(name, parts, c_p, c_w, seg=None, L=32768):
    offsets, xi = _csr(parts)
    C = len(c_p)
    return Workload(name, C, offsets, None if seg is None else np.asarray(seg, np.int32), xi,
                    np.full(C, L, np.int32), eta_grid(3, L), lam_grid(2), _f32(c_p), _f32(c_w), 1,
                    np.zeros(C, np.float32))


def _check(ctx, dev, w):
    import torch
    import paper_2607_16892_amd as dro
    print(f"[gpu] {w.name}: C={w.C} S={len(w.offsets) - 1} N={int(w.offsets[-1])}", flush=True)
    prob = dro.Problem.from_workload(w, dev)
    q = dro.class_quantile(ctx, prob)
    torch.cuda.synchronize()
    qv, qr = oracle.quantile(w)
    assert np.array_equal(q["q_rank"].cpu().numpy(), qr)
    got = q["q_value"].cpu().numpy()
    bad = np.flatnonzero(got != qv)
    assert bad.size == 0, f"q_value differs for classes {bad[:8]}: {got[bad[:8]]} vs {qv[bad[:8]]}"


def test_packed_halves_and_top_value(ctx, dev):
    # every class's segment puts its rank on a value next to a packing or
    # bucket edge: 0, 127/128, 16383/16384 (the half switch), 32767, 32768
    rng = np.random.default_rng(11)
    edges = [0, 1, 127, 128, 255, 16256, 16383, 16384, 16385, 16511, 16512, 32639, 32640, 32767,
             32768]
    parts, cps, cws = [], [], []
    for v in edges:
        for before in (0, 1, 5):
            # `before` samples below v (or at 0), one at v, the rest above (or at 2^15)
            lo = rng.integers(0, max(v, 1), before) if v > 0 else np.zeros(before, np.int64)
            hi = rng.integers(v, 32769, 7)
            parts.append(np.concatenate([lo, [v], hi]).astype(np.int32))
            # rank j = before + 1 exactly: c_p/(c_p+c_w) = (before + 1)/N, N = before + 8
            n = before + 8
            cps.append(float(before + 1))
            cws.append(float(n - before - 1))
    w = _workload("edges", parts, cps, cws)
    qv, _ = oracle.quantile(w)
    assert sorted(set(qv.tolist())) == edges  # the ranks land on the edge values
    _check(ctx, dev, w)


def test_uniform_full_range_ranks_at_bucket_edges(ctx, dev):
    # 2^15 + 1 samples: every value 0 .. 2^15 once, so rank j is the value j - 1;
    # the cost ratios put j on the first and last value of coarse buckets
    x = np.random.default_rng(12).permutation(np.arange(32769, dtype=np.int32))
    targets = [1, 128, 129, 256, 16384, 16385, 16512, 32640, 32641, 32768, 32769]
    N = 32769
    # c_p / (c_p + c_w) = (j - 1/2) / N, so ceil(c_p N / (c_p + c_w)) = j, with both
    # costs inside the accepted [2^-10, 2^7]
    cps, cws = [], []
    for j in targets:
        ratio = (j - 0.5) / (N - j + 0.5)
        cps.append(2.0 ** -10 * max(ratio, 1.0))
        cws.append(2.0 ** -10 / min(ratio, 1.0))
    w = _workload("uniform-edges", [x], cps, cws, seg=[0] * len(targets))
    qv, qr = oracle.quantile(w)
    assert list(qr) == targets and list(qv) == [j - 1 for j in targets]
    _check(ctx, dev, w)


@pytest.mark.parametrize("dist", ["constant", "lognormal", "top"])
def test_long_segments_need_more_blocks(ctx, dev, dist):
    # 300,001 and 131,071 samples per segment: each block holds at most 65,535
    # samples, so the segment is split further than one block per compute unit
    # would; constant samples put every count of a block on one packed half
    rng = np.random.default_rng(13)
    parts = []
    for n in (300_001, 131_071, 65_536, 1):
        if dist == "constant":
            x = np.full(n, 7, np.int32)
        elif dist == "top":
            x = np.full(n, 32768, np.int32)
        else:
            x = np.clip(np.rint(rng.lognormal(4.0, 1.5, n)), 1, 32768).astype(np.int32)
        parts.append(x)
    w = _workload(f"long-{dist}", parts, [8.0, 1.0, 3.0, 5.0], [1.0, 1.0, 1.0, 0.25])
    _check(ctx, dev, w)


def test_many_aliased_classes_and_extreme_ratios(ctx, dev):
    # 96 classes on 3 segments; cost ratios from 2^-17 (rank 1) to 2^17 (rank N)
    rng = np.random.default_rng(14)
    parts = [np.clip(np.rint(rng.lognormal(m, 1.0, n)), 1, 32768).astype(np.int32)
             for m, n in ((2.0, 5000), (6.0, 70_000), (9.0, 1))]
    C = 96
    r = np.linspace(-17, 17, C)
    c_p = _f32(np.where(r >= 0, 2.0 ** 7, 2.0 ** (7 + r)))
    c_w = _f32(np.where(r >= 0, 2.0 ** (7 - r), 2.0 ** 7))
    w = _workload("aliased", parts, c_p, c_w, seg=[c % 3 for c in range(C)])
    _, qr = oracle.quantile(w)
    n0 = 5000
    assert qr[0] == 1 and qr[C - 3] == n0  # class 0 and class 93 share segment 0
    _check(ctx, dev, w)


def test_repeated_calls_and_shrinking_problem(ctx, dev):
    # the per-block rows are scratch: a smaller problem after a larger one must
    # not read rows the larger one left behind
    rng = np.random.default_rng(15)
    big = _workload("big", [np.clip(np.rint(rng.lognormal(5, 1, 400_000)), 1, 32768)
                            .astype(np.int32) for _ in range(3)], [4.0, 9.0, 30.0],
                    [1.0, 1.0, 1.0])
    small = _workload("small", [np.clip(np.rint(rng.lognormal(3, 1, 900)), 1, 32768)
                                .astype(np.int32) for _ in range(2)], [2.0, 60.0], [1.0, 1.0])
    for w in (big, small, big, small):
        _check(ctx, dev, w)


@pytest.mark.parametrize("n_small,n_big", [(300, 3_000_001), (2000, 1 << 24)])
def test_segments_with_unequal_part_counts(ctx, dev, n_small, n_big):
    # one long segment among many short ones: the long one is split into
    # ceil(n / 65535) blocks, every short one takes one, and the rows of a
    # segment are found through the row table (with one count of blocks for
    # all segments, 2000 + 1 segments of up to 2^24 samples would need 514k rows)
    rng = np.random.default_rng(16 + n_small)
    parts = [rng.integers(1, 32769, int(rng.integers(1, 201))).astype(np.int32)
             for _ in range(n_small)]
    big = np.clip(np.rint(rng.lognormal(6.0, 1.4, n_big)), 1, 32768).astype(np.int32)
    big[::9973] = 32768
    mid = n_small // 2
    parts.insert(mid, big)
    S = len(parts)
    C = S + 99
    seg = [c % S for c in range(C)]
    seg[1] = seg[S] = seg[S + 7] = mid  # three more classes on the long segment
    r = rng.uniform(-17, 17, C)
    c_p = _f32(np.where(r >= 0, 2.0 ** 7, 2.0 ** (7 + r)))
    c_w = _f32(np.where(r >= 0, 2.0 ** (7 - r), 2.0 ** 7))
    w = _workload(f"unequal-{n_small}", parts, c_p, c_w, seg=seg)
    _check(ctx, dev, w)
