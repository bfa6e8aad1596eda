"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Stage by stage, each kernel is fed the same inputs as the oracle stage:
bitmaps and pool sizes, alpha and w_f, distance tables and the scan + top-k
must be bit-exact.  End to end from raw inputs: ids bit-exact, distances
bit-exact to the fp32 oracle and within 1e-4 relative of the fp64
definition."""
import numpy as np
import pytest
import torch

import oracle as O
from workload import make_workload, random_index
from tests._gpu_util import (assert_bitexact, check_search_row, oracle_from_workload,
                             oracle_index, say)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


@pytest.fixture(scope="module")
def c1(B):
    say("[c1] generating workload on cuda")
    w = make_workload("c1", device="cuda")
    idx = B.Index.from_workload(w, max_batch=128, max_k=128)
    return w, idx, oracle_from_workload(w)


def _np(t):
    return t.detach().cpu().numpy()


# ------------------------------------------------------------------ stages
def test_filter_bitmaps_and_counts_bitexact(B, c1):
    w, idx, ox = c1
    preds = w.preds[0.1]
    bm, cnt = idx.filter(preds)
    torch.cuda.synchronize()
    bm, cnt = _np(bm).view(np.uint32), _np(cnt)
    for i, p in enumerate(preds):
        mask = O.predicate_mask(ox["attrs"], p)
        assert np.array_equal(bm[i], O.selection_bitmap(mask)), i
        assert cnt[i] == mask.sum()


def test_condition_alpha_and_wf_bitexact(B, c1):
    w, idx, ox = c1
    s = 0.1
    alpha, wf = idx.select_codebook(w.queries, w.preds[s], w.w_z[s])
    torch.cuda.synchronize()
    alpha, wf = _np(alpha), _np(wf)
    for i in range(w.queries.shape[0]):
        a_o, wf_o = O.select_codebook(_np(w.queries[i]), w.preds[s][i], ox["bank"], ox["h"],
                                      ox["hash_seed"], _np(w.w_z[s][i]))
        assert_bitexact(alpha[i], a_o, f"alpha q{i}")
        assert_bitexact(wf[i], wf_o, f"w_f q{i}")
    # no w_z: w_f is exactly 1
    _, wf1 = idx.select_codebook(w.queries[:4], w.preds[s][:4], None)
    assert torch.all(wf1 == 1.0)


@pytest.mark.parametrize("conditioned", [True, False])
@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_lut_bitexact(B, c1, conditioned, dtype):
    w, idx, ox = c1
    s = 0.1
    lut_dt = B.LUT_F16 if dtype == "f16" else B.LUT_F32
    alpha, wf = idx.select_codebook(w.queries, w.preds[s], w.w_z[s])
    lut = idx.build_lut(w.queries, alpha if conditioned else None, wf, lut_dt)
    torch.cuda.synchronize()
    lut, alpha_h, wf_h = _np(lut), _np(alpha), _np(wf)
    for i in range(0, w.queries.shape[0], 7):
        ref = O.build_lut(_np(w.queries[i]), alpha_h[i] if conditioned else None, wf_h[i],
                          ox["C_pq"], ox["W"], w.M, w.r, lut_dtype=dtype)
        assert_bitexact(lut[i], ref, f"LUT {dtype} q{i}")


@pytest.mark.parametrize("dtype", ["f32", "f16"])
def test_scan_and_select_on_gpu_tables_bitexact(B, c1, dtype):
    """Rank + Select fed the GPU's own tables: ids and distances bit-exact."""
    w, idx, ox = c1
    s = 0.1
    lut_dt = B.LUT_F16 if dtype == "f16" else B.LUT_F32
    alpha, wf = idx.select_codebook(w.queries, w.preds[s], w.w_z[s])
    lut = idx.build_lut(w.queries, alpha, wf, lut_dt)
    ids, dist = idx.search(w.preds[s], lut, w.k, lut_dt)
    torch.cuda.synchronize()
    lut_h, ids, dist = _np(lut), _np(ids), _np(dist)
    for i, p in enumerate(w.preds[s]):
        cand = O.passing_ids(O.predicate_mask(ox["attrs"], p))
        d = O.adc_distances(lut_h[i], ox["codes"], cand)
        ids_o, dist_o = O.select_topk(d, cand, w.k)
        check_search_row(ids[i], dist[i], ids_o, dist_o, f"{dtype} q{i}")


@pytest.mark.parametrize("conditioned", [True, False])
def test_end_to_end_c1_from_raw_inputs(B, c1, conditioned):
    w, idx, ox = c1
    s = 0.1
    alpha, wf = idx.select_codebook(w.queries, w.preds[s], w.w_z[s])
    lut = idx.build_lut(w.queries, alpha if conditioned else None, wf)
    ids, dist, bm = idx.search(w.preds[s], lut, w.k, want_bitmap=True)
    torch.cuda.synchronize()
    ids, dist, bm = _np(ids), _np(dist), _np(bm).view(np.uint32)
    for i, p in enumerate(w.preds[s]):
        q, wz = _np(w.queries[i]), _np(w.w_z[s][i])
        res = O.filtered_search(ox, q, p, w.k, w_z=wz, conditioned=conditioned)
        res64 = O.filtered_search(ox, q, p, w.k, w_z=wz, conditioned=conditioned, dtype=np.float64)
        assert np.array_equal(bm[i], O.selection_bitmap(res["mask"]))
        check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"q{i}",
                         dist64=res64["dist"][: w.k])
        # every returned id passes the predicate
        good = ids[i][ids[i] >= 0]
        assert res["mask"][good].all()


# -------------------------------------------------------------- edge cases
def _edge_index(B, N, M, dsub, n_attr=2, domain=50, seed=0, conditioned=True, max_k=128,
                max_batch=64, cluster_cols=(), bank_rows=64, h=None):
    ix = random_index(N, M, dsub, n_attr, domain, seed, device="cuda", bank_rows=bank_rows)
    if h is not None:
        ix["h"] = h
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"] if conditioned else None,
                  ix["W"] if conditioned else None, ix["r"], ix["h"], ix["hash_seed"],
                  max_batch=max_batch, max_k=max_k, cluster_cols=cluster_cols)
    ox = oracle_index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"] if conditioned else None,
                      ix["W"] if conditioned else None, ix["r"], ix["h"], ix["hash_seed"])
    return idx, ox


def _run_and_check(B, idx, ox, preds, k, dsub, M, lut_dtype="f32", conditioned=True, seed=1):
    g = torch.Generator(device="cuda").manual_seed(seed)
    nq = len(preds)
    q = torch.randn(nq, M * dsub, device="cuda", generator=g)
    wz = 0.5413 + 0.3 * torch.randn(nq, M * dsub, device="cuda", generator=g)
    dt = B.LUT_F16 if lut_dtype == "f16" else B.LUT_F32
    alpha, wf = idx.select_codebook(q, preds, wz)
    lut = idx.build_lut(q, alpha if conditioned else None, wf, dt)
    ids, dist = idx.search(preds, lut, k, dt)
    torch.cuda.synchronize()
    ids, dist = _np(ids), _np(dist)
    for i, p in enumerate(preds):
        res = O.filtered_search(ox, _np(q[i]), p, k, w_z=_np(wz[i]), lut_dtype=lut_dtype,
                                conditioned=conditioned)
        check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"q{i} {p}")
    return ids


@pytest.mark.parametrize("N,M,dsub", [(1, 16, 8), (63, 16, 8), (65, 48, 2), (4097, 120, 8),
                                      (3000, 4, 3), (777, 7, 2), (20_001, 16, 8)])
def test_ragged_sizes_and_generic_m(B, N, M, dsub):
    say(f"[edge] N={N} M={M} dsub={dsub}")
    idx, ox = _edge_index(B, N, M, dsub, seed=N + M)
    preds = [[(0, 5, 40)], [(0, 0, 50), (1, 10, 30)], [], [(1, 7, 8)], [(0, 30, 10)]] * 3
    _run_and_check(B, idx, ox, preds, k=10, dsub=dsub, M=M)


@pytest.mark.parametrize("k", [1, 10, 64, 100, 300])
def test_k_range_including_pool_sorted_in_lds(B, k):
    say(f"[edge] k={k}")
    idx, ox = _edge_index(B, 30_000, 16, 8, seed=k, max_k=300)
    preds = [[(0, 0, 25)], [(0, 10, 11)], [(1, 0, 50)], [(0, 3, 4), (1, 3, 4)]] * 2
    _run_and_check(B, idx, ox, preds, k=k, dsub=8, M=16)


def test_pool_smaller_than_k_and_empty_pool(B):
    idx, ox = _edge_index(B, 5000, 16, 8, domain=1000, seed=3)
    preds = [[(0, 7, 8)], [(0, 7, 7)], [(0, 9, 3)], [(0, -(1 << 62), 1 << 62), (1, 999, 1000)]]
    ids = _run_and_check(B, idx, ox, preds, k=20, dsub=8, M=16)
    assert np.all(ids[1] == -1) and np.all(ids[2] == -1)


@pytest.mark.parametrize("cluster_cols", [(), (0,)])
def test_non_power_of_two_bank(B, cluster_cols):
    """B = 45,000 bank rows (a bank size of the paper's Table 2) with h = 3
    hash functions: alpha and w_f bit-exact, and the conditioned search from
    raw inputs equal to the oracle's."""
    say(f"[bank] B=45000 h=3 cluster={cluster_cols}")
    idx, ox = _edge_index(B, 20_000, 16, 8, n_attr=2, domain=1000, seed=45, bank_rows=45000, h=3,
                          cluster_cols=cluster_cols)
    rng = np.random.default_rng(45)
    preds = [[(0, int(lo), int(lo) + 100)] for lo in rng.integers(0, 900, 40)] + \
            [[(0, 5, 500), (1, 0, 300)], [], [(1, 17, 18)]]
    g = torch.Generator(device="cuda").manual_seed(46)
    q = torch.randn(len(preds), 128, device="cuda", generator=g)
    wz = 0.5413 + 0.1 * torch.randn(len(preds), 128, device="cuda", generator=g)
    alpha, wf = idx.select_codebook(q, preds, wz)
    torch.cuda.synchronize()
    alpha_h, wf_h = _np(alpha), _np(wf)
    masked_differs = 0
    for i, p in enumerate(preds):
        a_o, wf_o = O.select_codebook(_np(q[i]), p, ox["bank"], 3, ox["hash_seed"], _np(wz[i]))
        assert_bitexact(alpha_h[i], a_o, f"alpha q{i}")
        assert_bitexact(wf_h[i], wf_o, f"w_f q{i}")
        key = O.fingerprint(_np(q[i]), p)
        rows = O.hashed_rows(key, 3, 45000, ox["hash_seed"])
        masked = [O.splitmix64(key ^ O.splitmix64(ox["hash_seed"] + j)) & 44999 for j in range(3)]
        masked_differs += rows != masked
    assert masked_differs >= len(preds) - 1     # the modulus, not a bit mask, decides the rows
    _run_and_check(B, idx, ox, preds, k=10, dsub=8, M=16, seed=47)


def test_identity_index_and_fp16_tables(B):
    idx, ox = _edge_index(B, 12_345, 48, 2, conditioned=False, seed=5)
    preds = [[(0, 0, 20)], [(1, 5, 45)], []] * 5
    _run_and_check(B, idx, ox, preds, k=10, dsub=2, M=48, conditioned=False)
    _run_and_check(B, idx, ox, preds, k=10, dsub=2, M=48, conditioned=False, lut_dtype="f16")


@pytest.mark.parametrize("cluster_cols", [(), (0,)])
def test_ties_at_the_kth_distance_across_workgroups(B, cluster_cols):
    """Many rows share the k-th distance and sit in different wavefronts and
    workgroups (forced small chunks); the answer keeps the smallest ids."""
    ix = random_index(30_000, 48, 2, 1, 30, 43, device="cuda")
    ix["codes"][5::37] = ix["codes"][2]               # 811 copies of row 2
    ix["codes"][11::53] = ix["codes"][9]              # 566 copies of row 9
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=8, max_k=16, cluster_cols=cluster_cols)
    idx.set_option(B.OPT_SPLITS, 7)
    ox = oracle_index(ix["codes"], ix["C_pq"], ix["attrs"])
    C = ix["C_pq"]
    r2 = C[torch.arange(48, device="cuda"), ix["codes"][2].long()].reshape(-1)
    r9 = C[torch.arange(48, device="cuda"), ix["codes"][9].long()].reshape(-1)
    q = torch.stack([r2, r9, 0.5 * (r2 + r9), r2 + 0.01]).contiguous()
    preds = [[(0, 0, 30)], [(0, 3, 25)], [(0, 0, 30)], [(0, 10, 12)]]
    lut = idx.build_lut(q)
    for shared in (0, 1, 2):
        idx.set_option(B.OPT_SHARED_BOUND, shared)
        for k in (1, 10, 16):
            ids, dist = idx.search(preds, lut, k)
            torch.cuda.synchronize()
            for i, p in enumerate(preds):
                res = O.filtered_search(ox, _np(q[i]), p, k, conditioned=False)
                check_search_row(_np(ids[i]), _np(dist[i]), res["ids"], res["dist"], f"ties k={k} q{i} s{shared}")
    idx.set_option(B.OPT_SPLITS, 0)
    idx.set_option(B.OPT_SHARED_BOUND, 0)


def test_ties_broken_by_smaller_id(B):
    ix = random_index(4000, 16, 8, 1, 10, 11, device="cuda")
    ix["codes"][1000:1200] = ix["codes"][17]          # 201 identical rows
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=8, max_k=64)
    ox = oracle_index(ix["codes"], ix["C_pq"], ix["attrs"])
    rec = ix["C_pq"][torch.arange(16, device="cuda"), ix["codes"][17].long()].reshape(-1)
    q = rec[None].repeat(2, 1).contiguous()
    lut = idx.build_lut(q)
    ids, dist = idx.search([[], [(0, 0, 5)]], lut, 50)
    torch.cuda.synchronize()
    for i, p in enumerate([[], [(0, 0, 5)]]):
        res = O.filtered_search(ox, _np(q[i]), p, 50, conditioned=False)
        check_search_row(_np(ids[i]), _np(dist[i]), res["ids"], res["dist"], f"ties q{i}")
    assert _np(dist[0])[0] == 0.0 and list(_np(ids[0])[:3]) == [17, 1000, 1001]


def test_many_attribute_columns(B):
    idx, ox = _edge_index(B, 9000, 16, 8, n_attr=4, domain=20, seed=9)
    preds = [[(3, 2, 9)], [(2, 0, 10), (3, 5, 20), (0, 1, 19), (1, 0, 15)], [(2, 4, 5)]] * 3
    _run_and_check(B, idx, ox, preds, k=10, dsub=8, M=16)


@pytest.mark.parametrize("qtile,splits", [(1, 1), (2, 3), (3, 7), (8, 0), (6, 40)])
def test_forced_tiles_and_splits_same_answer(B, qtile, splits):
    idx, ox = _edge_index(B, 50_000, 16, 8, seed=21)
    idx.set_option(B.OPT_QTILE, qtile)
    idx.set_option(B.OPT_SPLITS, splits)
    preds = [[(0, 0, 25)], [(1, 3, 9)], [(0, 10, 12)]] * 5
    _run_and_check(B, idx, ox, preds, k=10, dsub=8, M=16)


def test_repeat_calls_are_deterministic(B, c1):
    w, idx, _ = c1
    s = 0.1
    outs = []
    for _ in range(3):
        alpha, wf = idx.select_codebook(w.queries, w.preds[s], w.w_z[s])
        lut = idx.build_lut(w.queries, alpha, wf)
        ids, dist = idx.search(w.preds[s], lut, w.k)
        torch.cuda.synchronize()
        outs.append((_np(ids), _np(dist).view(np.uint32)))
    for o in outs[1:]:
        assert np.array_equal(o[0], outs[0][0]) and np.array_equal(o[1], outs[0][1])


# ------------------------------------------------- clustered physical layout
@pytest.mark.parametrize("conditioned", [True, False])
def test_clustered_c1_matches_oracle(B, conditioned):
    """Rows stored in attribute order: same ids and distances as the oracle."""
    say("[clustered] c1")
    w = make_workload("c1", device="cuda")
    idx = B.Index.from_workload(w, max_batch=128, max_k=16, cluster_cols=(0,))
    ox = oracle_from_workload(w)
    s = 0.1
    alpha, wf = idx.select_codebook(w.queries, w.preds[s], w.w_z[s])
    lut = idx.build_lut(w.queries, alpha if conditioned else None, wf)
    ids, dist, bm = idx.search(w.preds[s], lut, w.k, want_bitmap=True)
    torch.cuda.synchronize()
    assert idx.last_plan()["qtile"] == 1
    ids, dist, bm = _np(ids), _np(dist), _np(bm).view(np.uint32)
    for i, p in enumerate(w.preds[s]):
        res = O.filtered_search(ox, _np(w.queries[i]), p, w.k, w_z=_np(w.w_z[s][i]),
                                conditioned=conditioned)
        assert np.array_equal(bm[i], O.selection_bitmap(res["mask"]))
        check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"q{i}")


@pytest.mark.parametrize("cols", [(0,), (1, 0), (0, 1), (2,)])
def test_clustered_predicate_shapes(B, cols):
    """Range, equality + range, rank prefix + range, residual clauses on other
    columns, predicates that miss the cluster key, contradictions."""
    say(f"[clustered] cols={cols}")
    idx, ox = _edge_index(B, 40_000, 16, 8, n_attr=3, domain=30, seed=31, cluster_cols=cols)
    preds = [
        [(0, 3, 9)], [(1, 7, 8), (0, 2, 20)], [(1, 0, 5), (0, 4, 25)], [(0, 5, 6), (1, 5, 6)],
        [(2, 1, 4)], [(2, 0, 10), (1, 3, 12), (0, 0, 28)], [], [(0, 9, 9)], [(0, 3, 9), (0, 10, 20)],
        [(1, -(1 << 40), 1 << 40), (0, 29, 1 << 50)], [(0, 0, 30), (0, 12, 13), (1, 2, 3)],
        [(1, 4, 5), (0, 17, 18), (2, 2, 29)],
    ] * 2
    _run_and_check(B, idx, ox, preds, k=10, dsub=8, M=16)
    _run_and_check(B, idx, ox, preds, k=100, dsub=8, M=16, seed=2)


@pytest.mark.parametrize("cols", [(0,), (0, 1)])
def test_clustered_wide_key_range(B, cols):
    """A leading cluster key whose values span ~3e7 integers (too wide for the
    value -> row table, so every interval bound comes from the 64-ary search)
    and, for comparison, the same rows with a narrow key (table lookups):
    both give the oracle's results."""
    say(f"[clustered] wide key cols={cols}")
    S, OFF = 1_000_003, -(1 << 30)
    base = [[(0, 3, 9)], [(0, 7, 8), (1, 2, 20)], [(0, 0, 30)], [(0, 29, 30)], [(0, 12, 12)],
            [(0, -5, 2)], [(0, 28, 1 << 20)], [(0, 5, 6), (1, 5, 6)], [(1, 3, 7)], []]
    for wide in (True, False):
        ix = random_index(20_000, 16, 8, 2, 30, 43, device="cuda")
        preds = base
        if wide:
            ix["attrs"][0] = ix["attrs"][0] * S + OFF
            preds = [[(c, lo * S + OFF, hi * S + OFF) if c == 0 else (c, lo, hi) for c, lo, hi in p]
                     for p in base]
        idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"],
                      ix["hash_seed"], max_batch=16, max_k=32, cluster_cols=cols)
        ox = oracle_index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"],
                          ix["hash_seed"])
        _run_and_check(B, idx, ox, preds, k=32, dsub=8, M=16)


@pytest.mark.parametrize("cols", [(0,), (1, 0)])
def test_clustered_chunk_grid_and_fallback(B, cols):
    """Chunks cut on a grid of cells (forced small here; long spans get one by
    default), including spans that need more cells than there are chunks
    (cut into equal chunks instead): results equal the default plan's, which
    equal the oracle's."""
    say(f"[clustered] chunk grid cols={cols}")
    idx, ox = _edge_index(B, 40_000, 16, 8, n_attr=2, domain=30, seed=37, cluster_cols=cols)
    a, b = cols[0], 1 - cols[0]          # a: the cluster key every predicate bounds
    preds = [[(a, 3, 9)], [(a, 0, 30)], [(a, 7, 8), (b, 2, 20)], [(a, 11, 12)], [(a, 1, 27), (b, 0, 15)],
             [(a, 29, 30), (b, 2, 9)], [(a, 1, 27)], [(a, -5, 100)]] * 3
    g = torch.Generator(device="cuda").manual_seed(3)
    q = torch.randn(len(preds), 128, device="cuda", generator=g)
    alpha, wf = idx.select_codebook(q, preds, None)
    lut = idx.build_lut(q, alpha, wf)
    ids0, dist0 = idx.search(preds, lut, 20)
    torch.cuda.synchronize()
    assert idx.last_plan()["grid_tiles"] == 0          # spans too short for a grid by default
    for i, p in enumerate(preds[:8]):
        lut_o = O.build_lut(_np(q[i]), _np(alpha[i]), _np(wf[i]), ox["C_pq"], ox["W"], 16, ox["r"])
        cand = O.passing_ids(O.predicate_mask(ox["attrs"], p))
        ids_o, dist_o = O.select_topk(O.adc_distances(lut_o, ox["codes"], cand), cand, 20)
        check_search_row(_np(ids0[i]), _np(dist0[i]), ids_o, dist_o, f"grid q{i}")
    # absolute cells (64-tile grid: one chunk per cell fits), relative cells,
    # and grids whose cells outnumber the chunks (equal-chunk fallback); for
    # absolute cells both dispatch orders (estimated work, index order)
    for grid, splits, relative, order in ((64, 0, 0, 0), (64, 0, 0, 1), (64, 0, 1, 0), (100, 0, 0, 0),
                                          (1, 0, 0, 0), (1, 0, 0, 1), (7, 0, 1, 0), (7, 2, 0, 0),
                                          (1, 3, 1, 0), (64, 1, 0, 0), (13, 0, 0, 0)):
        idx.set_option(B.OPT_GRID_TILES, grid)
        idx.set_option(B.OPT_SPLITS, splits)
        idx.set_option(B.OPT_GRID_RELATIVE, relative)
        idx.set_option(B.OPT_SLOT_ORDER, order)
        ids, dist = idx.search(preds, lut, 20)
        torch.cuda.synchronize()
        assert idx.last_plan()["grid_tiles"] == grid
        assert torch.equal(ids, ids0), (grid, splits, relative, order)
        assert torch.equal(dist.view(torch.int32), dist0.view(torch.int32)), (grid, splits, relative, order)
    idx.set_option(B.OPT_GRID_TILES, 0)
    idx.set_option(B.OPT_SPLITS, 0)
    idx.set_option(B.OPT_GRID_RELATIVE, 0)
    idx.set_option(B.OPT_SLOT_ORDER, 0)
    # k = 10: grid scans turn on the workgroup bound (published best keys)
    ids10, dist10 = idx.search(preds, lut, 10)
    torch.cuda.synchronize()
    assert torch.equal(ids10, ids0[:, :10]) and torch.equal(dist10.view(torch.int32), dist0[:, :10].view(torch.int32))
    for grid, shared in ((64, 0), (1, 0), (13, 1), (0, 2)):
        idx.set_option(B.OPT_GRID_TILES, grid)
        idx.set_option(B.OPT_SHARED_BOUND, shared)
        ids, dist = idx.search(preds, lut, 10)
        torch.cuda.synchronize()
        assert torch.equal(ids, ids10), (grid, shared)
        assert torch.equal(dist.view(torch.int32), dist10.view(torch.int32)), (grid, shared)
    idx.set_option(B.OPT_GRID_TILES, 0)
    idx.set_option(B.OPT_SHARED_BOUND, 0)


@pytest.mark.parametrize("cluster_cols,M,dsub,k,lut_dtype", [((), 16, 8, 10, "f32"), ((), 48, 2, 100, "f32"),
                                                         ((), 16, 8, 37, "f16"), ((1,), 48, 2, 10, "f32")])
def test_gather_scan_matches_oracle(B, cluster_cols, M, dsub, k, lut_dtype):
    """Masked batches: queries scored from their compacted row lists (forced
    on, automatic, forced off) give the oracle's ids and distance bits, with
    pools from empty to the whole index."""
    say(f"[gather] cols={cluster_cols} M={M} k={k} {lut_dtype}")
    idx, ox = _edge_index(B, 30_000, M, dsub, n_attr=2, domain=40, seed=53, cluster_cols=cluster_cols)
    preds = [[(0, 3, 4)], [(0, 0, 40)], [(1, 5, 7), (0, 2, 30)], [], [(0, 9, 9)], [(1, 0, 1), (0, 39, 40)],
             [(0, 10, 30)], [(1, 17, 18)], [(0, 5, 6), (1, 5, 6)], [(1, 0, 20)]] * 2
    g = torch.Generator(device="cuda").manual_seed(7)
    q = torch.randn(len(preds), M * dsub, device="cuda", generator=g)
    dt = B.LUT_F16 if lut_dtype == "f16" else B.LUT_F32
    alpha, wf = idx.select_codebook(q, preds, None)
    lut = idx.build_lut(q, alpha, wf, dt)
    outs = {}
    for mode in (1, 0, 2):
        idx.set_option(B.OPT_GATHER, mode)
        ids, dist = idx.search(preds, lut, k, dt)
        torch.cuda.synchronize()
        outs[mode] = (_np(ids), _np(dist))
    idx.set_option(B.OPT_GATHER, 0)
    for i, p in enumerate(preds[:10]):
        lut_o = O.build_lut(_np(q[i]), _np(alpha[i]), _np(wf[i]), ox["C_pq"], ox["W"], M, ox["r"],
                            lut_dtype=lut_dtype)
        cand = O.passing_ids(O.predicate_mask(ox["attrs"], p))
        ids_o, dist_o = O.select_topk(O.adc_distances(lut_o.astype(np.float32), ox["codes"], cand), cand, k)
        for mode, (ids, dist) in outs.items():
            check_search_row(ids[i], dist[i], ids_o, dist_o, f"gather={mode} q{i} {p}")
    for mode in (0, 2):
        assert np.array_equal(outs[mode][0], outs[1][0])
        assert np.array_equal(outs[mode][1].view(np.uint32), outs[1][1].view(np.uint32))


def test_gather_compaction_sparse_and_dense_workgroups(B):
    """Row lists of gather-mode queries over several compaction workgroups
    (65536 rows each): pools that a workgroup stages in LDS (about 1% and 5%
    of its rows) and pools too large for that (about 20%), which it writes
    directly; the search gives the oracle's ids and distance bits either way
    and matches the tiled scan."""
    say("[gather] compaction paths N=150000")
    idx, ox = _edge_index(B, 150_000, 16, 8, n_attr=1, domain=100, seed=61, max_k=16)
    preds = [[(0, 50, 51)], [(0, 0, 5)], [(0, 10, 30)], [(0, 93, 100)], [(0, 7, 8)], [(0, 60, 80)]]
    idx.set_option(B.OPT_GATHER, 1)
    ids = _run_and_check(B, idx, ox, preds, k=16, dsub=8, M=16)
    idx.set_option(B.OPT_GATHER, 2)
    ids2 = _run_and_check(B, idx, ox, preds, k=16, dsub=8, M=16)
    idx.set_option(B.OPT_GATHER, 0)
    assert np.array_equal(ids, ids2)


@pytest.mark.parametrize("k", [200, 16, 10])
def test_clustered_ties_break_by_original_id(B, k):
    """Equal rows everywhere: the k-th distance is shared by many rows of
    every wavefront, so the workgroup bound (k <= 16) and the deferred id
    lookup must still keep the smaller original ids."""
    ix = random_index(6000, 16, 8, 1, 40, 41, device="cuda")
    ix["codes"][::7] = ix["codes"][3]                 # equal rows in every cluster
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=8, max_k=200, cluster_cols=(0,))
    ox = oracle_index(ix["codes"], ix["C_pq"], ix["attrs"])
    rec = ix["C_pq"][torch.arange(16, device="cuda"), ix["codes"][3].long()].reshape(-1)
    q = rec[None].repeat(3, 1).contiguous()
    preds = [[], [(0, 10, 30)], [(0, 5, 6)]]
    lut = idx.build_lut(q)
    ids, dist = idx.search(preds, lut, k)
    torch.cuda.synchronize()
    for i, p in enumerate(preds):
        res = O.filtered_search(ox, _np(q[i]), p, k, conditioned=False)
        check_search_row(_np(ids[i]), _np(dist[i]), res["ids"], res["dist"], f"ties q{i}")
    # interval batches with a seeded bound: the seed's k-th distance is the
    # shared one, and rows at it must still be decided by original id
    iv_preds = preds[1:]
    ids0, dist0 = idx.search(iv_preds, lut[1:], k)
    for seed_tiles in (2, 24):
        idx.set_option(B.OPT_SEED_TILES, seed_tiles)
        ids1, dist1 = idx.search(iv_preds, lut[1:], k)
        torch.cuda.synchronize()
        assert torch.equal(ids1, ids0) and torch.equal(dist1.view(torch.int32), dist0.view(torch.int32)), seed_tiles
    idx.set_option(B.OPT_SEED_TILES, 0)


def test_clustered_and_plain_layouts_agree_on_c4_sample(B):
    """A 1M-row slice of the 10M-vector workload: both layouts, every bin."""
    say("[clustered] c4 slice")
    w = make_workload("c4", device="cuda", N=1_000_000, n_queries=64, keep_x=False)
    plain = B.Index.from_workload(w, max_batch=64, max_k=10)
    clus = B.Index.from_workload(w, max_batch=64, max_k=10, cluster_cols=(0,))
    for s in w.bins:
        a, f = plain.select_codebook(w.queries, w.preds[s], w.w_z[s])
        lut = plain.build_lut(w.queries, a, f)
        i1, d1 = plain.search(w.preds[s], lut, 10)
        i2, d2 = clus.search(w.preds[s], lut, 10)
        torch.cuda.synchronize()
        assert torch.equal(i1, i2), s
        assert torch.equal(d1.view(torch.int32), d2.view(torch.int32)), s
        # seeded bounds (mixture data: the seed is close to the answer)
        for seed_tiles in (1, 2, 24, 48):
            clus.set_option(B.OPT_SEED_TILES, seed_tiles)
            i3, d3 = clus.search(w.preds[s], lut, 10)
            torch.cuda.synchronize()
            assert torch.equal(i1, i3), (s, seed_tiles)
            assert torch.equal(d1.view(torch.int32), d3.view(torch.int32)), (s, seed_tiles)
        clus.set_option(B.OPT_SEED_TILES, 0)


@pytest.mark.parametrize("cluster_cols", [(), (0,)])
def test_negative_weights_rank_exactly(B, cluster_cols):
    """Caller-supplied weights may be negative: table entries and distances
    go negative, partial sums stop being lower bounds, and the ranking must
    still match the oracle bit for bit."""
    idx, ox = _edge_index(B, 20_000, 48, 2, seed=77, cluster_cols=cluster_cols)
    g = torch.Generator(device="cuda").manual_seed(5)
    preds = [[(0, 0, 40)], [(0, 10, 20)], [(1, 5, 45)], []] * 2
    q = torch.randn(len(preds), 96, device="cuda", generator=g)
    wf = torch.randn(len(preds), 96, device="cuda", generator=g)          # mixed signs
    alpha, _ = idx.select_codebook(q, preds, None)
    lut = idx.build_lut(q, alpha, wf)
    ids, dist = idx.search(preds, lut, 25)
    torch.cuda.synchronize()
    for i, p in enumerate(preds):
        lut_o = O.build_lut(_np(q[i]), _np(alpha[i]), _np(wf[i]), ox["C_pq"], ox["W"], 48, ox["r"])
        cand = O.passing_ids(O.predicate_mask(ox["attrs"], p))
        ids_o, dist_o = O.select_topk(O.adc_distances(lut_o, ox["codes"], cand), cand, 25)
        check_search_row(_np(ids[i]), _np(dist[i]), ids_o, dist_o, f"neg q{i}")
    assert (dist < 0).any()
    if cluster_cols:
        # no seed where partial sums are no bound (the table has negative entries)
        iv = [p for p in preds if p]
        ids0, dist0 = idx.search(iv, lut[[i for i, p in enumerate(preds) if p]], 25)
        idx.set_option(B.OPT_SEED_TILES, 24)
        ids1, dist1 = idx.search(iv, lut[[i for i, p in enumerate(preds) if p]], 25)
        torch.cuda.synchronize()
        idx.set_option(B.OPT_SEED_TILES, 0)
        assert torch.equal(ids1, ids0) and torch.equal(dist1.view(torch.int32), dist0.view(torch.int32))


@pytest.mark.parametrize("cols,M,dsub", [((0,), 16, 8), ((1, 0), 16, 8), ((0,), 48, 2), ((0,), 120, 8)])
def test_seeded_bound_same_answer(B, cols, M, dsub):
    """The seeded bound (a k-th distance over candidate rows ranked by their
    first subspace group) on short intervals (tiles drawn from the whole
    interval: all of them, or evenly spaced ones) and on chunk-grid cells,
    with residual clauses, empty intervals, k up to 64 (and 65, where no seed
    is taken): every setting gives the unseeded answer, which is the
    oracle's."""
    say(f"[seed] cols={cols} M={M}")
    idx, ox = _edge_index(B, 30_000, M, dsub, n_attr=2, domain=30, seed=53 + M, cluster_cols=cols)
    a, b = cols[0], 1 - cols[0]
    preds = [[(a, 3, 9)], [(a, 0, 30)], [(a, 7, 8), (b, 2, 20)], [(a, 11, 12)], [(a, 1, 27), (b, 0, 15)],
             [(a, 29, 30)], [(a, 9, 9)], [(a, 4, 26)]] * 2
    g = torch.Generator(device="cuda").manual_seed(M)
    q = torch.randn(len(preds), M * dsub, device="cuda", generator=g)
    alpha, wf = idx.select_codebook(q, preds, None)
    lut = idx.build_lut(q, alpha, wf)
    lut16 = idx.build_lut(q, alpha, wf, B.LUT_F16)
    for k in (1, 10, 64, 65):
        idx.set_option(B.OPT_SEED_TILES, 1)
        ids0, dist0 = idx.search(preds, lut, k)
        i16, d16 = idx.search(preds, lut16, k, B.LUT_F16)
        torch.cuda.synchronize()
        if k == 10:
            for i, p in enumerate(preds[:8]):
                lut_o = O.build_lut(_np(q[i]), _np(alpha[i]), _np(wf[i]), ox["C_pq"], ox["W"], M, ox["r"])
                cand = O.passing_ids(O.predicate_mask(ox["attrs"], p))
                ids_o, dist_o = O.select_topk(O.adc_distances(lut_o, ox["codes"], cand), cand, k)
                check_search_row(_np(ids0[i]), _np(dist0[i]), ids_o, dist_o, f"seed q{i} {p}")
        for seed_tiles, grid in ((2, 0), (3, 0), (24, 0), (1000, 0), (0, 64), (2, 64), (24, 7), (0, 1)):
            idx.set_option(B.OPT_SEED_TILES, seed_tiles)
            idx.set_option(B.OPT_GRID_TILES, grid)
            ids, dist = idx.search(preds, lut, k)
            torch.cuda.synchronize()
            assert torch.equal(ids, ids0), (k, seed_tiles, grid)
            assert torch.equal(dist.view(torch.int32), dist0.view(torch.int32)), (k, seed_tiles, grid)
            if seed_tiles in (2, 24):                    # binary16 tables
                ids, dist = idx.search(preds, lut16, k, B.LUT_F16)
                torch.cuda.synchronize()
                assert torch.equal(ids, i16) and torch.equal(dist.view(torch.int32), d16.view(torch.int32))
    idx.set_option(B.OPT_SEED_TILES, 0)
    idx.set_option(B.OPT_GRID_TILES, 0)


@pytest.mark.parametrize("seed_tiles", [0, 8])
def test_clustered_batch_with_unsatisfiable_predicates(B, seed_tiles):
    """Predicates no row satisfies (lo >= hi, contradictory ranges) have the
    empty interval on a clustered index: the batch keeps the one-query
    interval plan and those rows come back as padding, the rest as the
    oracle's."""
    say(f"[edge] clustered batch with empty predicates seed={seed_tiles}")
    idx, ox = _edge_index(B, 40_000, 48, 2, n_attr=1, domain=500, seed=71, cluster_cols=(0,))
    idx.set_option(B.OPT_SEED_TILES, seed_tiles)
    preds = [[(0, 10, 60)], [(0, 9, 9)], [(0, 100, 400)], [(0, 30, 20)], [(0, 5, 50), (0, 70, 90)],
             [(0, 0, 500)], [(0, 499, 500)]] * 3
    ids = _run_and_check(B, idx, ox, preds, k=10, dsub=2, M=48)
    assert idx.last_plan()["qtile"] == 1
    for i, p in enumerate(preds):
        if i % 7 in (1, 3, 4):
            assert np.all(ids[i] == -1), p
    idx.set_option(B.OPT_SEED_TILES, 0)
