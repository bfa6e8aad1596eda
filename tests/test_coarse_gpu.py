"""The coarse bound of the Rank stage (ifvs_build_coarse, ifvs_lut_bounds,
ifvs_filtered_search_bounded): an exact pruning device, so every result must
equal the plain search's, bit for bit, and the oracle's.

Pins of the pieces, checked on the CPU in fp64 against their definitions:
* every stored radius bounds ||C_PQ(x) - C_PQ(centroid)|| from above (and
  is that distance rounded up to a bfloat16), and the assigned centroid is a
  nearest encoded one;
* the per-query factors bound sqrt(max w_f) and delta = sqrt(sum over m of
  (2 max_c ||Delta[m][c]||)^2) from above, delta computed from the oracle's
  conditioned codebook;
* the bound itself holds for every row of several queries: sqrt(dist) >=
  sqrt(dist to its centroid) - sqrt(max w) (r + delta), distances summed in
  fp64 over the GPU's tables.
Then the search: structured data (10%, 50% intervals, k from 1 to 100),
fp32 and binary16 tables, conditioned, identity and SDC tables, residual
clauses, negative weights (bound off), unsatisfiable predicates, exact ties
at the k-th distance."""
import numpy as np
import pytest
import torch

import oracle as O
from workload import make_workload
from tests._gpu_util import check_search_row, oracle_from_workload, oracle_index, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


def _np(t):
    return t.detach().cpu().numpy()


@pytest.fixture(scope="module")
def c4s(B):
    """120K rows of the 96-d, 48 x 2 workload, clustered by its attribute."""
    say("[coarse] c4 sample N=120000")
    w = make_workload("c4", device="cuda", N=120_000, n_queries=48, keep_x=False)
    idx = B.Index.from_workload(w, max_batch=64, max_k=128, cluster_cols=(0,))
    idx.build_coarse(256, 10)
    return w, idx, oracle_from_workload(w)


def _recon(codes, C_pq):
    M = codes.shape[1]
    return np.concatenate([C_pq[m][codes[:, m].astype(np.int64)] for m in range(M)], axis=1).astype(np.float64)


def test_build_is_deterministic_and_radii_bound_the_distance(B, c4s):
    w, idx, ox = c4s
    assign, radius, cc = idx.read_coarse()
    assert cc.shape == (256, 48) and assign.shape == (w.N,)
    assert assign.min() >= 0 and assign.max() < 256
    idx.build_coarse(256, 10)
    a2, r2, c2 = idx.read_coarse()
    assert np.array_equal(a2, assign) and np.array_equal(r2.view(np.uint32), radius.view(np.uint32))
    assert np.array_equal(c2, cc)
    # radii: the fp64 distance to the assigned centroid, rounded up to bf16
    X = _recon(ox["codes"], ox["C_pq"])
    Cr = _recon(cc, ox["C_pq"])
    exact = np.sqrt(((X - Cr[assign]) ** 2).sum(1))
    r = radius.astype(np.float64)
    assert np.all(r >= exact), "a stored radius is below the distance it bounds"
    assert np.all(r <= exact * (1 + 2.0 ** -14) * (1 + 2.0 ** -7) * (1 + 1e-6) + 1e-30)
    assert np.all((radius.view(np.uint32) & 0xFFFF) == 0)
    # the assigned centroid is a nearest one (rows sampled)
    rows = np.arange(0, w.N, 97)
    d = ((X[rows, None, :] - Cr[None]) ** 2).sum(-1)
    assert np.all(d[np.arange(rows.size), assign[rows]] <= d.min(1) * (1 + 1e-5) + 1e-12)


def test_build_arguments(B, c4s):
    w, idx, ox = c4s
    for bad in ((0, 1), (4097, 1), (16, -1), (16, 1001)):
        with pytest.raises(B.IfvsError) as e:
            idx.build_coarse(*bad)
        assert e.value.status == B.E_INVALID
    tiny = B.Index(w.codes[:100], w.C_pq, w.attrs[:, :100], max_batch=4, max_k=4)
    with pytest.raises(B.IfvsError):
        tiny.build_coarse(101, 1)            # more centroids than rows
    with pytest.raises(B.IfvsError) as e:
        tiny.read_coarse()
    assert e.value.status == B.E_STATE
    tiny.build_coarse(100, 0)                # every row is a centroid; no iteration
    a, r, _ = tiny.read_coarse()
    assert np.all(r == 0.0)
    tiny.close()


def test_lut_bounds_pin_sqrt_wmax_and_delta(B, c4s):
    w, idx, ox = c4s
    nq = 16
    q = w.queries[:nq]
    wz = w.w_z[0.1][:nq]
    alpha, wf = idx.select_codebook(q, w.preds[0.1][:nq], wz)
    b = _np(idx.lut_bounds(nq, alpha, wf)).astype(np.float64)
    wf_n, al = _np(wf).astype(np.float64), _np(alpha)
    for i in range(nq):
        sw = np.sqrt(wf_n[i].max())
        assert sw <= b[i, 0] <= sw * (1 + 1e-5)
        # the shift of the fp32 conditioned codewords the tables are built
        # from, taken exactly (fp64 difference of fp32 values)
        Cc = O.conditioned_codebook(ox["C_pq"], ox["W"], al[i], w.M, ox["r"], dtype=np.float32)
        dl = Cc.astype(np.float64) - ox["C_pq"].astype(np.float64)     # [M][256][dsub]
        delta = np.sqrt((4.0 * (dl ** 2).sum(-1).max(-1)).sum())
        assert delta <= b[i, 1] <= delta * (1 + 1e-5), (i, delta, b[i, 1])
    # no conditioning: delta 0; no weights: sqrt(max w) = 1 (widened)
    b0 = _np(idx.lut_bounds(nq, None, None))
    assert np.all(b0[:, 1] == 0.0) and np.all((b0[:, 0] >= 1.0) & (b0[:, 0] <= 1.0 + 1e-5))
    # a negative or non-finite weight switches the bound off (NaN)
    wf_bad = wf.clone()
    wf_bad[0, 3] = -0.5
    wf_bad[1, 7] = float("inf")
    wf_bad[2, 0] = float("nan")
    bb = _np(idx.lut_bounds(nq, alpha, wf_bad))
    assert np.all(np.isnan(bb[:3, 0])) and np.all(np.isfinite(bb[3:, 0]))
    st = B.lib().ifvs_lut_bounds(idx.handle, nq, alpha.data_ptr(), wf.data_ptr(), None, None)
    assert st == B.E_INVALID


def test_bound_holds_for_every_row(B, c4s):
    """sqrt(d(x)) >= sqrt(d(c)) - sqrt(max w) (r_x + delta) for all 120K rows
    of 6 conditioned queries, in fp64 over the GPU's own tables."""
    w, idx, ox = c4s
    nq = 6
    q = w.queries[:nq]
    alpha, wf = idx.select_codebook(q, w.preds[0.5][:nq], w.w_z[0.5][:nq])
    lut = _np(idx.build_lut(q, alpha, wf)).astype(np.float64)
    bnd = _np(idx.lut_bounds(nq, alpha, wf)).astype(np.float64)
    assign, radius, cc = idx.read_coarse()
    codes = ox["codes"].astype(np.int64)
    m_idx = np.arange(w.M)
    pruned = 0
    for i in range(nq):
        d = lut[i][m_idx, codes].sum(1)
        dc = lut[i][m_idx, cc.astype(np.int64)].sum(1)
        lb = np.sqrt(dc)[assign] - bnd[i, 0] * (radius.astype(np.float64) + bnd[i, 1])
        # the tables hold fp32 roundings of the exact distances
        assert np.all(np.sqrt(d) >= lb - 1e-6 * (np.sqrt(d) + np.sqrt(dc)[assign])), i
        kth = np.sort(d)[9]
        pruned += int(np.sum((lb > 0) & (lb * lb > kth)))
    say(f"[coarse] rows the bound prunes at the final 10th distance: {pruned / (nq * w.N):.3f}")
    assert pruned > 0


def _search_pair(B, idx, preds, lut, alpha, wf, k, dt):
    idx.set_option(B.OPT_COARSE, 1)
    ids0, d0 = idx.search(preds, lut, k, dt)
    idx.set_option(B.OPT_COARSE, 2)
    ids1, d1 = idx.search_bounded(preds, lut, alpha, wf, k, dt)
    torch.cuda.synchronize()
    used = idx.last_coarse()
    idx.set_option(B.OPT_COARSE, 0)
    assert torch.equal(ids1, ids0) and torch.equal(d1.view(torch.int32), d0.view(torch.int32))
    return _np(ids1), _np(d1), used


@pytest.mark.parametrize("lut_dtype", ["f32", "f16"])
@pytest.mark.parametrize("mode", ["conditioned", "identity", "sdc"])
def test_bounded_search_equals_plain_and_oracle(B, c4s, lut_dtype, mode):
    w, idx, ox = c4s
    dt = B.LUT_F16 if lut_dtype == "f16" else B.LUT_F32
    nq = 24
    for s in (0.1, 0.5):
        preds = w.preds[s][:nq]
        q = w.queries[:nq]
        wz = w.w_z[s][:nq]
        if mode == "sdc":
            lut = idx.build_sdc_lut(q, dt)
            a = wf = None
        else:
            alpha, wf = idx.select_codebook(q, preds, wz)
            a = alpha if mode == "conditioned" else None
            lut = idx.build_lut(q, a, wf, dt)
        for k in (1, 10, 100):
            say(f"[coarse] {mode} {lut_dtype} s={s} k={k}")
            ids, dist, used = _search_pair(B, idx, preds, lut, a, wf, k, dt)
            assert used
            if k == 10:
                for i in range(0, nq, 3):
                    if mode == "sdc":
                        res = O.sdc_filtered_search(ox, _np(q[i]), preds[i], k, lut_dtype=lut_dtype)
                    else:
                        res = O.filtered_search(ox, _np(q[i]), preds[i], k, w_z=_np(wz[i]), lut_dtype=lut_dtype,
                                                conditioned=mode == "conditioned")
                    check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"{mode} s={s} q{i}")


def test_auto_mode(B):
    """Automatic mode: the list scan for a batch whose widest interval spans
    8192 or more tiles, the interval scan for short intervals; the plain
    search never takes it.  Answers identical throughout."""
    say("[coarse] automatic mode, 640K rows")
    w = make_workload("c4", device="cuda", N=640_000, n_queries=8, keep_x=False)
    idx = B.Index.from_workload(w, max_batch=8, max_k=16, cluster_cols=(0,))
    idx.build_coarse(512, 4)
    nq = 8
    preds = [[(0, 0, 3650)]] * nq          # every row: a span of 10K tiles
    q = w.queries[:nq]
    alpha, wf = idx.select_codebook(q, preds, w.w_z[0.5][:nq])
    lut = idx.build_lut(q, alpha, wf)
    ids0, d0 = idx.search(preds, lut, 10)
    assert not idx.last_coarse()
    ids1, d1 = idx.search_bounded(preds, lut, alpha, wf, 10)
    assert idx.last_coarse()
    short = [[(0, 100, 110)]] * nq                          # 0.3% of the rows
    ids2, d2 = idx.search_bounded(short, lut, alpha, wf, 10)
    assert not idx.last_coarse()
    ids3, d3 = idx.search(short, lut, 10)
    torch.cuda.synchronize()
    assert torch.equal(ids1, ids0) and torch.equal(d1.view(torch.int32), d0.view(torch.int32))
    assert torch.equal(ids2, ids3) and torch.equal(d2.view(torch.int32), d3.view(torch.int32))
    idx.close()


def test_negative_weights_unsatisfiable_predicates_and_residual_clauses(B):
    """Two attribute columns, rows clustered by (category, range value).
    Batch 1, every selection a row interval (equality on the category and a
    range, or the category alone, or nothing; some unsatisfiable), some
    queries with negative weights (tables with negative entries: no early
    abandonment and no bound): the list scan runs and matches the oracle.
    Batch 2 adds a clause on the minor column alone (tested row by row): the
    plain scan runs, with the same answers as without the bounds."""
    say("[coarse] two columns, negative weights, empty predicates, residual clauses")
    w = make_workload("c2", device="cuda", N=60_000, n_queries=24, keep_x=False)
    idx = B.Index.from_workload(w, max_batch=32, max_k=64, cluster_cols=(1, 0))
    idx.build_coarse(128, 8)
    ox = oracle_from_workload(w)
    batch1 = [[(0, 100, 800), (1, 2, 3)], [(1, 0, 1)], [(1, 5, 5)], [(0, 50, 950), (1, 3, 4)],
              [(1, 2, 3), (1, 5, 6)], [], [(1, 0, 100)]] * 3
    batch2 = [[(0, 100, 800)], [(0, 0, 1000), (1, 0, 5)], [(1, 7, 8)], [(0, 300, 400), (1, 1, 2)]] * 4
    for bi, (preds, listed) in enumerate(((batch1, True), (batch2, False))):
        nq = len(preds)
        q = w.queries[:nq]
        alpha, wf = idx.select_codebook(q, preds, w.w_z[0.1][:nq])
        wf = wf.clone()
        wf[1::5, 0] = -1.0
        lut = idx.build_lut(q, alpha, wf)
        ids, dist, used = _search_pair(B, idx, preds, lut, alpha, wf, 10, B.LUT_F32)
        assert used == listed
        alpha_n, wf_n = _np(alpha), _np(wf)
        for i in range(nq):
            lut_o = O.build_lut(_np(q[i]), alpha_n[i], wf_n[i], ox["C_pq"], ox["W"], w.M, ox["r"])
            cand = O.passing_ids(O.predicate_mask(ox["attrs"], preds[i]))
            ids_o, dist_o = O.select_topk(O.adc_distances(lut_o, ox["codes"], cand), cand, 10)
            check_search_row(ids[i], dist[i], ids_o, dist_o, f"batch{bi} q{i} {preds[i]}")
    idx.close()


@pytest.mark.parametrize("lut_dtype", ["f32", "f16"])
def test_ties_at_the_kth_distance(B, lut_dtype):
    """Most rows share one of 3 code vectors (and so a centroid and a
    radius): distances tie in large groups at the k-th place.  The bound
    must keep every row of the tie (the smallest ids win)."""
    say(f"[coarse] ties {lut_dtype}")
    g = torch.Generator(device="cuda").manual_seed(5)
    N, M, dsub = 50_000, 48, 2
    C_pq = torch.randn(M, 256, dsub, device="cuda", generator=g)
    base = torch.randint(0, 256, (3, M), device="cuda", generator=g, dtype=torch.int64)
    pick = torch.randint(0, 3, (N,), device="cuda", generator=g)
    codes = base[pick].to(torch.uint8)
    noisy = torch.rand(N, device="cuda", generator=g) < 0.02
    codes[noisy] = torch.randint(0, 256, (int(noisy.sum()), M), device="cuda", generator=g,
                                 dtype=torch.int64).to(torch.uint8)
    attrs = torch.randint(0, 100, (1, N), device="cuda", generator=g, dtype=torch.int32)
    idx = B.Index(codes.contiguous(), C_pq, attrs, max_batch=16, max_k=128, cluster_cols=(0,))
    idx.build_coarse(8, 4)
    ox = oracle_index(codes, C_pq, attrs)
    dt = B.LUT_F16 if lut_dtype == "f16" else B.LUT_F32
    # queries at the first code vector's reconstruction (distance 0 ties) and near it
    rec = torch.stack([C_pq[m, base[0, m]] for m in range(M)]).reshape(-1)
    q = rec[None].repeat(8, 1) + torch.cat([torch.zeros(4, M * dsub, device="cuda"),
                                            0.01 * torch.randn(4, M * dsub, device="cuda", generator=g)])
    preds = [[(0, 0, 100)], [(0, 10, 90)], [(0, 0, 50)], [(0, 20, 100)]] * 2
    lut = idx.build_lut(q, None, None, dt)
    for k in (5, 64, 128):
        ids, dist, used = _search_pair(B, idx, preds, lut, None, None, k, dt)
        assert used
        for i in range(8):
            res = O.filtered_search(ox, _np(q[i]), preds[i], k, lut_dtype=lut_dtype, conditioned=False)
            check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"ties k={k} q{i}")
    idx.close()


def test_m16_index(B):
    say("[coarse] 128-d, 16 x 8 index")
    w = make_workload("c2", device="cuda", N=100_000, n_queries=16, keep_x=False)
    idx = B.Index.from_workload(w, max_batch=16, max_k=16, cluster_cols=(1, 0))
    idx.build_coarse(512, 10)
    ox = oracle_from_workload(w)
    # (at 50% the category clause is a prefix of categories and the range
    # clause is tested row by row: not a list-scan batch)
    for s in (0.01, 0.1):
        preds = w.preds[s][:16]
        q = w.queries[:16]
        alpha, wf = idx.select_codebook(q, preds, w.w_z[s][:16])
        lut = idx.build_lut(q, alpha, wf)
        ids, dist, used = _search_pair(B, idx, preds, lut, alpha, wf, 10, B.LUT_F32)
        assert used
        for i in range(0, 16, 4):
            res = O.filtered_search(ox, _np(q[i]), preds[i], 10, w_z=_np(w.w_z[s][i]))
            check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"m16 s={s} q{i}")
    idx.close()


def test_counting_build_of_the_list_scan(B, c4s):
    """The list scan's read-counting build: same answers as the timed build;
    it sums at least one tile, reads every tile's first groups and the rest
    of at most every tile, and its table reads come in groups of eight
    subspaces (M = 48)."""
    w, idx, ox = c4s
    nq = 24
    s = 0.5
    preds = w.preds[s][:nq]
    q = w.queries[:nq]
    alpha, wf = idx.select_codebook(q, preds, w.w_z[s][:nq])
    lut = idx.build_lut(q, alpha, wf)
    idx.set_option(B.OPT_COARSE, 2)
    try:
        ids0, d0 = idx.search_bounded(preds, lut, alpha, wf, 10)
        idx.set_option(B.OPT_COUNT_READS, 1)
        idx.read_scan_reads()
        ids1, d1 = idx.search_bounded(preds, lut, alpha, wf, 10)
        torch.cuda.synchronize()
        assert idx.last_coarse()
        hist = idx.read_scan_reads()
    finally:
        idx.set_option(B.OPT_COUNT_READS, 0)
        idx.set_option(B.OPT_COARSE, 0)
    assert torch.equal(ids1, ids0) and torch.equal(d1.view(torch.int32), d0.view(torch.int32))
    assert len(hist) == 66
    assert hist[0] > 0 and 0 <= hist[65] <= hist[0]
    assert sum(hist[1:65]) % 8 == 0
    assert sum(hist[1:65]) >= 8 * hist[0]   # every tile reads its first group
