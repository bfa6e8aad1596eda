"""ifvs_query_batch, the whole path of Section 2 in one call (encoder,
condition, tables, bounded search), against the same stages called one by
one: every output (w_z, alpha, w_f, the tables, ids, distance bits) equal
bit for bit, with and without a given w_z, fp32 and binary16 tables, list
scan forced on (the table kernel then also writes the bound's factors), the
condition inside the encoder's launch (h of 1 to 4, no bank) or in its own
kernel (h = 5); then a sample of rows against the oracle, and the error
paths (each leaves the index usable)."""
import numpy as np
import pytest
import torch

import oracle as O
from workload import random_encoder, random_index
from tests._gpu_util import check_search_row, oracle_index, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


@pytest.fixture(scope="module")
def case(B):
    """40K rows, M = 48 subspaces of 2 dims, a bank of 97 rows, clustered by
    the first of two attributes, a 64-centroid coarse build and an encoder."""
    say("[query_batch] index N=40000 M=48")
    M, dsub = 48, 2
    ix = random_index(40_000, M, dsub, 2, 1000, seed=17, device="cuda", bank_rows=97)
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], ix["hash_seed"],
                  max_batch=64, max_k=32, cluster_cols=(0,))
    idx.load_encoder(random_encoder(2, M * dsub, [1000, 1000], seed=4))
    idx.build_coarse(64, 5)
    g = torch.Generator(device="cpu").manual_seed(8)
    nq = 40
    q = torch.randn(nq, M * dsub, generator=g).cuda()
    preds = []
    for i in range(nq):
        lo = int(torch.randint(0, 900, (1,), generator=g))
        w = [0, 1, 30, 100, 500, 1000][i % 6]
        preds.append([(0, lo, lo + w)] + ([(1, 100, 700)] if i % 7 == 3 else []))
    return ix, idx, q, preds


def _bits(t):
    return t.contiguous().view(torch.int32) if t.dtype == torch.float32 else t.contiguous().view(torch.int16)


def _stagewise(idx, q, preds, k, w_z, lut_dtype):
    wz = idx.encode_predicates(preds) if w_z is None else w_z
    alpha, wf = idx.select_codebook(q, preds, wz)
    lut = idx.build_lut(q, alpha, wf, lut_dtype)
    ids, dist = idx.search_bounded(preds, lut, alpha, wf, k, lut_dtype)
    return ids, dist, wz, alpha, wf, lut


@pytest.mark.parametrize("given_wz", [False, True])
@pytest.mark.parametrize("lut_dtype", [0, 1])
@pytest.mark.parametrize("mode", [0, 2])
def test_same_bits_as_the_separate_calls(B, case, given_wz, lut_dtype, mode):
    ix, idx, q, preds = case
    say(f"[query_batch] given_wz={given_wz} lut_dtype={lut_dtype} coarse_mode={mode}")
    k = 20
    w_z = None
    if given_wz:
        w_z = torch.rand(q.shape[0], q.shape[1], device="cuda", generator=torch.Generator(device="cuda")
                         .manual_seed(3)) * 0.5 + 0.25
    # residual clauses take the batch off the list scan: drop them in forced mode
    p = [c[:1] for c in preds] if mode == 2 else preds
    idx.set_option(B.OPT_COARSE, mode)
    try:
        ref = _stagewise(idx, q, p, k, w_z, lut_dtype)
        used_ref = idx.last_coarse()
        got = idx.query_batch(q, p, k, w_z=w_z, lut_dtype=lut_dtype)
        used = idx.last_coarse()
    finally:
        idx.set_option(B.OPT_COARSE, 0)
    torch.cuda.synchronize()
    assert used == used_ref and used == (mode == 2)
    for name, a, b in zip(("ids", "dist", "w_z", "alpha", "w_f", "lut"), got, ref):
        assert a.shape == b.shape, name
        assert torch.equal(_bits(a) if a.is_floating_point() else a, _bits(b) if b.is_floating_point() else b), name


@pytest.mark.parametrize("h,bank_rows", [(1, 45), (3, 97), (4, 1000), (5, 33), (0, 0)])
def test_condition_in_the_encoder_launch(B, h, bank_rows):
    """The encoder launch conditions the queries itself for h <= 4 (and
    without a bank); h = 5 takes the condition kernel.  Either way alpha,
    w_f, the tables and the results are the separate calls' bits."""
    say(f"[query_batch] h={h} bank_rows={bank_rows}")
    M, dsub = 16, 4
    ix = random_index(9_000, M, dsub, 2, 300, seed=h + 40, device="cuda", bank_rows=max(bank_rows, 1))
    bank, W = (ix["bank"], ix["W"]) if bank_rows else (None, None)
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], bank, W, ix["r"] if bank_rows else 0, h,
                  ix["hash_seed"], max_batch=32, max_k=10, cluster_cols=(0,))
    idx.load_encoder(random_encoder(2, M * dsub, [300, 300], seed=h, layers=1))
    g = torch.Generator(device="cpu").manual_seed(h)
    q = torch.randn(29, M * dsub, generator=g).cuda()
    preds = [[(0, 7 * i, 7 * i + 40)] + ([(1, 0, 150)] if i % 3 == 0 else []) for i in range(29)]
    got = idx.query_batch(q, preds, 10)
    ref = _stagewise(idx, q, preds, 10, None, 0)
    torch.cuda.synchronize()
    for name, a, b in zip(("ids", "dist", "w_z", "alpha", "w_f", "lut"), got, ref):
        if a is None or b is None:
            assert a is None and b is None and name == "alpha"
            continue
        assert torch.equal(_bits(a) if a.is_floating_point() else a, _bits(b) if b.is_floating_point() else b), name


def test_chunk_grid_dispatch_order_from_the_encoder_launch(B):
    """An interval-scan batch wide enough for the chunk grid (>= 8192 tiles):
    the scan's dispatch order is copied to the device by the encoder's side
    workgroups under ifvs_query_batch, by the interval kernel otherwise; the
    results are the separate calls' bits either way."""
    say("[query_batch] chunk grid, N=600000")
    M, dsub = 16, 2
    ix = random_index(600_000, M, dsub, 1, 1000, seed=23, device="cuda", bank_rows=45)
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], ix["hash_seed"],
                  max_batch=16, max_k=10, cluster_cols=(0,))
    idx.load_encoder(random_encoder(1, M * dsub, [1000], seed=6, layers=1))
    g = torch.Generator(device="cpu").manual_seed(11)
    q = torch.randn(12, M * dsub, generator=g).cuda()
    preds = [[(0, 5 * i, 1000)] for i in range(12)]              # 94-100% of the rows each
    got = idx.query_batch(q, preds, 10)
    plan = idx.last_plan()
    ref = _stagewise(idx, q, preds, 10, None, 0)
    torch.cuda.synchronize()
    assert plan["grid_tiles"] > 0, plan                          # the chunk grid ran
    assert not idx.last_coarse()
    for name, a, b in zip(("ids", "dist", "w_z", "alpha", "w_f", "lut"), got, ref):
        assert torch.equal(_bits(a) if a.is_floating_point() else a, _bits(b) if b.is_floating_point() else b), name
    idx.set_option(B.OPT_SLOT_ORDER, 1)                          # the plain order: no copy at all
    ids2, dist2, *_ = idx.query_batch(q, preds, 10)
    idx.set_option(B.OPT_SLOT_ORDER, 0)
    torch.cuda.synchronize()
    assert torch.equal(ids2, ref[0]) and torch.equal(_bits(dist2), _bits(ref[1]))


def test_profile_mode_three_times_the_list_scan_only(B, case):
    ix, idx, q, preds = case
    p = [c[:1] for c in preds]
    for coarse, launches in ((2, 1), (1, 0)):           # list scan forced, then off
        idx.set_option(B.OPT_COARSE, coarse)
        idx.set_option(B.OPT_PROFILE, 3)
        idx.read_profile()
        idx.query_batch(q, p, 10)
        prof = idx.read_profile()
        idx.set_option(B.OPT_PROFILE, 0)
        idx.set_option(B.OPT_COARSE, 0)
        assert prof["scan"][1] == launches, (coarse, prof)
        assert all(n == 0 for st, (_, n) in prof.items() if st != "scan"), prof


def test_rows_against_the_oracle(B, case):
    ix, idx, q, preds = case
    say("[query_batch] oracle rows")
    k = 10
    p = [c[:1] for c in preds]
    idx.set_option(B.OPT_COARSE, 2)
    try:
        ids, dist, wz, *_ = idx.query_batch(q, p, k)
        assert idx.last_coarse()
    finally:
        idx.set_option(B.OPT_COARSE, 0)
    torch.cuda.synchronize()
    ox = oracle_index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], ix["hash_seed"])
    ids, dist, wz_h, q_h = ids.cpu().numpy(), dist.cpu().numpy(), wz.cpu().numpy(), q.cpu().numpy()
    for i in range(0, len(p), 5):
        res = O.filtered_search(ox, q_h[i], p[i], k, w_z=wz_h[i])
        check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"q{i} {p[i]}")


def test_errors_leave_the_index_usable(B, case):
    ix, idx, q, preds = case
    say("[query_batch] errors")
    with pytest.raises(B.IfvsError):
        idx.query_batch(q, preds, 33)                          # beyond max_k
    with pytest.raises(B.IfvsError):
        idx.query_batch(q, preds[:-1] + [[(5, 0, 1)]], 10)     # unknown attribute column
    q2 = torch.randn(65, q.shape[1], device="cuda")
    with pytest.raises(B.IfvsError):
        idx.query_batch(q2, [[]] * 65, 10)                     # beyond max_batch
    bare = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], ix["hash_seed"],
                   max_batch=8, max_k=10)
    with pytest.raises(B.IfvsError) as e:
        bare.query_batch(q[:2], preds[:2], 5)                  # no encoder, no w_z
    assert e.value.status == B.E_STATE
    empty = bare.query_batch(q[:0], [], 5)
    assert empty[0].shape == (0, 5)
    # the slots the failed calls staged were released
    for _ in range(6):
        ids, dist, *_ = idx.query_batch(q, preds, 10)
    ref = _stagewise(idx, q, preds, 10, None, 0)
    torch.cuda.synchronize()
    assert torch.equal(ids, ref[0]) and torch.equal(_bits(dist), _bits(ref[1]))
