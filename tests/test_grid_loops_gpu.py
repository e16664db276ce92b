"""Launches whose size grows with the problem loop over their items or rows
with at most 2^20 blocks (so a grid stays below 2^32 work-items).  These tests
take each loop past one pass, against the oracle's exact definitions:

- dro_argmin_reservation on C K = 4.7e6 rows (the minimum over the
  multipliers: 4 rows per block, two passes) and E C = 2^20 + 6 radius rows
  (the argmin, one block per row, two passes), from an exact S table drawn
  with many ties (App. A Step 3, Prop. 4.2; ties to the lowest k, then m);
- class_quantile on 2^20 + 5 classes (the select, one block per class);
- dro_cost_eval on a C K M = 268,500,992-entry table, past the 2^28 items
  of one pass of the zero fill and the exact epilogue, checked at sampled
  entries that include the last ones (App. A Steps 4-5).
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


def _costs(rng, C):
    choice = [(8.0, 1.0), (1.0, 1.0), (2.0 ** 7, 2.0 ** -10), (2.0 ** -10, 2.0 ** 7), (0.5, 3.0)]
    pick = rng.integers(len(choice), size=C)
    return _f32([choice[i][0] for i in pick]), _f32([choice[i][1] for i in pick])


def test_argmin_rows_past_one_pass(ctx, dev):
    import torch
    import paper_2607_16892_amd as dro
    rng = np.random.default_rng(31)
    C, K, M, E, L = (1 << 19) + 3, 9, 2, 2, 1000
    offsets, xi = _csr([rng.integers(0, L + 1, 3).astype(np.int32),
                        rng.integers(0, L + 1, 5).astype(np.int32)])
    seg = (np.arange(C) % 2).astype(np.int32)
    c_p, c_w = _costs(rng, C)
    eps = _f32(rng.uniform(0.0, 50.0, E * C))
    eps[:C] = 0.0
    w = Workload("rows", C, offsets, seg, xi, np.full(C, L, np.int32), eta_grid(K, L),
                 lam_grid(M, 0.5, 8.0), c_p, c_w, E, eps)
    assert C * K > 4 << 20 and E * C > 1 << 20
    # an exact S table (units of 2^-33) with ties: values from a small set
    lo = (rng.integers(0, 64, (C, K, M)).astype(np.uint64) << np.uint64(36))
    S = oracle.ExactS(np.zeros((C, K, M), np.int64), lo)
    Sd = S.to_double()
    print(f"[gpu] argmin rows: C={C} K={K} M={M} E={E}", flush=True)
    prob = dro.Problem.from_workload(w, dev)
    a = dro.dro_argmin_reservation(ctx, prob, torch.from_numpy(eps).to(dev),
                                   torch.from_numpy(Sd).to(dev))
    torch.cuda.synchronize()
    Wr, msr = oracle.W_table(w, S)
    ks, ws = oracle.argmin(Wr)
    assert np.array_equal(a["k_star"].cpu().numpy(), ks)
    assert np.array_equal(a["W_star"].cpu().numpy().view(np.uint64), ws.view(np.uint64))
    e_i, c_i = np.meshgrid(np.arange(E), np.arange(C), indexing="ij")
    assert np.array_equal(a["m_at_star"].cpu().numpy(), msr[e_i, c_i, ks])


def test_quantile_classes_past_one_pass(ctx, dev):
    rng = np.random.default_rng(32)
    C, L = (1 << 20) + 5, 32768
    parts = [rng.integers(1, L + 1, n).astype(np.int32) for n in (50, 1, 77)]
    offsets, xi = _csr(parts)
    seg = (np.arange(C) % 3).astype(np.int32)
    c_p, c_w = _costs(rng, C)
    w = Workload("classes", C, offsets, seg, xi, np.full(C, L, np.int32), eta_grid(3, L),
                 lam_grid(2), c_p, c_w, 1, np.zeros(C, np.float32))
    import torch
    import paper_2607_16892_amd as dro
    print(f"[gpu] quantile classes: C={C}", flush=True)
    q = dro.class_quantile(ctx, dro.Problem.from_workload(w, dev))
    torch.cuda.synchronize()
    qv, qr = oracle.quantile(w)
    assert np.array_equal(q["q_rank"].cpu().numpy(), qr)
    assert np.array_equal(q["q_value"].cpu().numpy(), qv)


def test_cost_eval_table_past_one_pass(ctx, dev):
    import torch
    import paper_2607_16892_amd as dro
    rng = np.random.default_rng(33)
    C, K, M, E, L = 32, 4097, 2048, 1, 4096
    offsets, xi = _csr([rng.integers(0, L + 1, 3).astype(np.int32),
                        np.array([0, L, 17], np.int32)])
    seg = (np.arange(C) % 2).astype(np.int32)
    c_p, c_w = _costs(rng, C)
    eps = _f32(rng.uniform(0.0, 30.0, E * C))
    w = Workload("table", C, offsets, seg, xi, np.full(C, L, np.int32), eta_grid(K, L),
                 lam_grid(M, 2.0 ** -10, 2.0 ** 7), c_p, c_w, E, eps)
    n = C * K * M
    assert n > (1 << 20) * 256
    print(f"[gpu] cost eval table: C={C} K={K} M={M} ({n} entries)", flush=True)
    prob = dro.Problem.from_workload(w, dev)
    r = dro.dro_cost_eval(ctx, prob, torch.from_numpy(eps).to(dev))
    torch.cuda.synchronize()
    Sg = r["S"].view(-1)
    # sampled entries, the last 4096 of the table among them
    idx = np.unique(np.concatenate([rng.integers(0, n, 3000), np.arange(n - 4096, n)]))
    cs, ks, ms = idx // (K * M), (idx // M) % K, idx % M
    ref = oracle.S_exact_at(w, cs, ks, ms).to_double()
    got = Sg[torch.from_numpy(idx).to(dev)].cpu().numpy()
    assert np.array_equal(got.view(np.uint64), ref.view(np.uint64))
    # whole W rows for a few (c, k), one of them the last
    Wg = r["W"].cpu().numpy()
    mg = r["m_star"].cpu().numpy()
    for c, k in ((0, 0), (7, 2048), (C - 1, K - 1)):
        S_row = oracle.S_exact_at(w, np.full(M, c), np.full(M, k), np.arange(M))
        N = int(offsets[seg[c] + 1] - offsets[seg[c]])
        J = [oracle.J(S_row.hi[m], S_row.lo[m], float(w.lam[m]), float(eps[c]), N) for m in range(M)]
        m_best = int(np.argmin(J))  # first index of the minimum
        assert Wg[0, c, k] == J[m_best] and mg[0, c, k] == m_best
