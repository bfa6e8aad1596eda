"""Exact filtered kNN on the GPU (ifvs_load_vectors / ifvs_exact_search)
against the CPU oracle: ids and distance bits equal on every query, for both
plans (direct exact scoring; matrix-core screening followed by exact
scoring), both row layouts, residual clauses, empty pools, pools smaller
than k, ties, ragged dimensions, the 10M-vector workload by sampling, and
the same search over the reconstructions of the codes."""
import numpy as np
import pytest
import torch

import oracle as O
from workload import make_workload, random_index
from tests._gpu_util import check_search_row, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


def _np(t):
    return t.detach().cpu().numpy()


def _index(B, N, D, n_attr=2, domain=40, seed=0, cluster_cols=(), max_batch=64, max_k=128, x=None):
    """A code-only index (codes are irrelevant to the exact search) plus
    Gaussian-mixture vectors attached with ifvs_load_vectors."""
    M = 8 if D % 8 == 0 else 1
    ix = random_index(N, M, D // M, n_attr, domain, seed, device="cuda")
    g = torch.Generator(device="cuda").manual_seed(seed + 1)
    if x is None:
        means = torch.rand(16, D, device="cuda", generator=g) * 2 - 1
        comp = torch.randint(0, 16, (N,), device="cuda", generator=g)
        x = means[comp] + 0.3 * torch.randn(N, D, device="cuda", generator=g)
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=max_batch, max_k=max_k,
                  cluster_cols=cluster_cols)
    idx.load_vectors(x)
    return idx, x, ix["attrs"]


def _check(B, idx, x, attrs, q, preds, k, what):
    ids, dist = idx.exact_search(q, preds, k)
    torch.cuda.synchronize()
    ids, dist = _np(ids), _np(dist)
    xh, ah = _np(x), _np(attrs)
    for i, p in enumerate(preds):
        res = O.exact_filtered_search(xh, ah, _np(q[i]), p, k)
        check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"{what} q{i} {p}")
    return ids, dist


def _queries(N, D, nq, seed, x):
    g = torch.Generator(device="cuda").manual_seed(seed)
    rows = torch.randint(0, N, (nq,), device="cuda", generator=g)
    return (x[rows] + 0.2 * torch.randn(nq, D, device="cuda", generator=g)).contiguous()


@pytest.mark.parametrize("plan", [0, 1, 2])
@pytest.mark.parametrize("cluster_cols", [(), (0,), (1, 0)])
def test_exact_search_matches_oracle(B, plan, cluster_cols):
    say(f"[exact] plan={plan} cols={cluster_cols}")
    N, D = 30_000, 96
    idx, x, attrs = _index(B, N, D, seed=3, cluster_cols=cluster_cols)
    idx.set_option(B.OPT_EXACT_PLAN, plan)
    preds = [[(0, 0, 40)], [(0, 5, 9)], [(0, 10, 30), (1, 3, 20)], [(1, 7, 8)], [],
             [(0, 30, 10)], [(0, 2, 3), (1, 2, 3)], [(0, 0, 20)]] * 5
    q = _queries(N, D, len(preds), 11, x)
    _check(B, idx, x, attrs, q, preds, 10, f"plan{plan}")
    idx.set_option(B.OPT_EXACT_PLAN, 0)


@pytest.mark.parametrize("D", [1, 40, 128, 200])
def test_exact_search_ragged_dimensions(B, D):
    say(f"[exact] D={D}")
    N = 5_003
    idx, x, attrs = _index(B, N, D, seed=D)
    preds = [[(0, 0, 40)], [(0, 3, 17)], [(1, 11, 12)]] * 4
    q = _queries(N, D, len(preds), D + 5, x)
    for plan in (1, 2):
        idx.set_option(B.OPT_EXACT_PLAN, plan)
        _check(B, idx, x, attrs, q, preds, 16, f"D{D} plan{plan}")
    idx.set_option(B.OPT_EXACT_PLAN, 0)


@pytest.mark.parametrize("k", [1, 64, 128])
def test_exact_search_k_range_and_small_pools(B, k):
    N, D = 12_000, 128
    idx, x, attrs = _index(B, N, D, seed=k, cluster_cols=(0,), domain=1000)
    preds = [[(0, 0, 1000)], [(0, 500, 520)], [(0, 7, 8)], [(0, 9, 9)], [(0, 100, 400), (1, 0, 3)]]
    q = _queries(N, D, len(preds), 50 + k, x)
    for plan in (1, 2):
        idx.set_option(B.OPT_EXACT_PLAN, plan)
        ids, _ = _check(B, idx, x, attrs, q, preds, k, f"k{k} plan{plan}")
        assert np.all(ids[3] == -1)
    idx.set_option(B.OPT_EXACT_PLAN, 0)


@pytest.mark.parametrize("cluster_cols", [(), (0,)])
def test_exact_search_ties_keep_smaller_ids(B, cluster_cols):
    """Hundreds of identical vectors at the k-th distance, spread over the
    index: every plan returns the smallest ids."""
    N, D = 20_000, 96
    g = torch.Generator(device="cuda").manual_seed(9)
    x = torch.randn(N, D, device="cuda", generator=g)
    x[3::29] = x[7]
    x[5::31] = x[11]
    idx, x, attrs = _index(B, N, D, seed=9, cluster_cols=cluster_cols, x=x)
    q = torch.stack([x[7], x[11], 0.5 * (x[7] + x[11]), x[7] + 1e-3]).contiguous()
    preds = [[(0, 0, 40)], [(0, 10, 30)], [], [(0, 5, 6)]]
    for plan in (1, 2):
        idx.set_option(B.OPT_EXACT_PLAN, plan)
        for k in (1, 10, 100):
            ids, dist = _check(B, idx, x, attrs, q, preds, k, f"ties plan{plan} k{k}")
    idx.set_option(B.OPT_EXACT_PLAN, 0)
    assert dist[0][0] == 0.0


def test_exact_search_overflowing_candidate_list_falls_back(B):
    """A query with more rows inside the screening bound than a candidate list
    holds (identical rows) is scored over its whole interval instead."""
    N, D = 40_000, 64
    x = torch.zeros(N, D, device="cuda")
    x[::2] = 1.0                       # 20000 identical rows, all at the k-th distance
    idx, x, attrs = _index(B, N, D, seed=4, x=x, domain=3)
    idx.set_option(B.OPT_EXACT_PLAN, 2)
    q = torch.ones(2, D, device="cuda")
    _check(B, idx, x, attrs, q, [[], [(0, 1, 2)]], 10, "overflow")
    idx.set_option(B.OPT_EXACT_PLAN, 0)


def test_exact_search_errors(B):
    from tests.test_abi_gpu import _status   # reuse: status and message of a raw call
    ix = random_index(1000, 8, 4, 1, 10, 1, device="cuda")
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=4, max_k=8)
    lib = B.lib()
    q = torch.zeros(1, 32, device="cuda")
    ids = torch.empty(1, 8, device="cuda", dtype=torch.int32)
    dist = torch.empty(1, 8, device="cuda")
    st, msg = _status(B, lib.ifvs_exact_search, idx.handle, 1, q.data_ptr(), B.pack_predicates([[]]), 8,
                      ids.data_ptr(), dist.data_ptr(), None)
    assert st == B.E_STATE, msg
    bad = torch.randn(1000, 32, device="cuda")
    bad[17, 3] = float("nan")
    st, msg = _status(B, lib.ifvs_load_vectors, idx.handle, bad.data_ptr(), B.MEM_DEVICE)
    assert st == B.E_INVALID and "NaN" in msg, msg
    good = torch.randn(1000, 32)
    idx.load_vectors(good)                          # host memory
    st, msg = _status(B, lib.ifvs_load_vectors, idx.handle, good.data_ptr(), B.MEM_HOST)
    assert st == B.E_STATE, msg
    for kk in (0, 9):
        st, _ = _status(B, lib.ifvs_exact_search, idx.handle, 1, q.data_ptr(), B.pack_predicates([[]]), kk,
                        ids.data_ptr(), dist.data_ptr(), None)
        assert st == B.E_INVALID
    st, _ = _status(B, lib.ifvs_exact_search, idx.handle, 5, q.data_ptr(), B.pack_predicates([[]] * 5), 8,
                    ids.data_ptr(), dist.data_ptr(), None)
    assert st == B.E_INVALID
    st, _ = _status(B, lib.ifvs_set_option, idx.handle, B.OPT_EXACT_PLAN, 3)
    assert st == B.E_INVALID
    # host-loaded vectors search like device-loaded ones
    ids2, dist2 = idx.exact_search(good[:3].cuda(), [[], [(0, 2, 5)], [(0, 9, 10)]], 8)
    torch.cuda.synchronize()
    for i, p in enumerate([[], [(0, 2, 5)], [(0, 9, 10)]]):
        res = O.exact_filtered_search(good.numpy(), _np(ix["attrs"]), good[i].numpy(), p, 8)
        check_search_row(_np(ids2[i]), _np(dist2[i]), res["ids"], res["dist"], f"host q{i}")


def test_exact_search_c4_10m_sampled(B):
    """The 10M-vector workload, 256-query batches, every bin: the oracle
    recomputes two queries per bin one by one."""
    say("[exact] generating c4 with its vectors")
    w = make_workload("c4", device="cuda", n_queries=256, keep_x=True)
    idx = B.Index.from_workload(w, max_batch=256, max_k=10, cluster_cols=(0,))
    idx.load_vectors(w.x)
    xh, ah = _np(w.x), _np(w.attrs)
    for s in w.bins:
        say(f"[exact] c4 bin {s}")
        ids, dist = idx.exact_search(w.queries, w.preds[s], 10)
        torch.cuda.synchronize()
        ids, dist = _np(ids), _np(dist)
        for i in (0, 131):
            res = O.exact_filtered_search(xh, ah, _np(w.queries[i]), w.preds[s][i], 10)
            check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"c4 s={s} q{i}")


@pytest.mark.parametrize("cluster_cols", [(), (0,)])
@pytest.mark.parametrize("plan", [1, 2])
def test_reconstruct_then_exact_matches_oracle(B, cluster_cols, plan):
    """Exact search over the reconstructions of the codes (the
    reconstruct-then-exact baseline) against the oracle's reconstruct +
    exact_filtered_search."""
    say(f"[exact] reconstructions cols={cluster_cols} plan={plan}")
    w = make_workload("c1", device="cuda", n_queries=40)
    idx = B.Index.from_workload(w, max_batch=40, max_k=w.k, cluster_cols=cluster_cols)
    idx.load_reconstructions()
    idx.set_option(B.OPT_EXACT_PLAN, plan)
    xh = O.reconstruct(_np(w.codes), _np(w.C_pq))
    preds = w.preds[w.bins[0]][:36] + [[], [(0, 3, 3)], [(0, 0, 1000)], [(0, 500, 501)]]
    ids, dist = idx.exact_search(w.queries, preds, w.k)
    torch.cuda.synchronize()
    ids, dist = _np(ids), _np(dist)
    for i, p in enumerate(preds):
        res = O.exact_filtered_search(xh, _np(w.attrs), _np(w.queries[i]), p, w.k)
        check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"rec q{i} {p}")
    st = B.lib().ifvs_load_reconstructions(idx.handle)
    assert st == B.E_STATE
