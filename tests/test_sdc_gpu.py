"""Symmetric distance computation on the GPU (ifvs_build_sdc_lut, then the
shared scan and top-k) against the CPU oracle: the per-query tables bit for
bit in fp32 and binary16, and whole searches (ids and distance bits) on both
row layouts and odd shapes."""
import numpy as np
import pytest
import torch

import oracle as O
from workload import make_workload, random_index
from tests._gpu_util import assert_bitexact, check_search_row, oracle_index, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


def _np(t):
    return t.detach().cpu().numpy()


@pytest.mark.parametrize("M,dsub", [(16, 8), (48, 2), (7, 3), (120, 8)])
def test_sdc_tables_bitexact(B, M, dsub):
    say(f"[sdc] tables M={M} dsub={dsub}")
    ix = random_index(3000, M, dsub, 1, 10, M + dsub, device="cuda")
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=16, max_k=10)
    g = torch.Generator(device="cuda").manual_seed(M)
    q = torch.randn(12, M * dsub, device="cuda", generator=g)
    q[3] = ix["C_pq"][torch.arange(M, device="cuda"), ix["codes"][5].long()].reshape(-1)   # a reconstruction
    T = O.sdc_table(_np(ix["C_pq"]))
    for dt, name in ((B.LUT_F32, "f32"), (B.LUT_F16, "f16")):
        lut = _np(idx.build_sdc_lut(q, dt))
        for i in range(q.shape[0]):
            ref = O.sdc_lut(_np(q[i]), _np(ix["C_pq"]), lut_dtype=name, table=T)
            assert_bitexact(lut[i], ref, f"sdc {name} q{i}")


@pytest.mark.parametrize("cluster_cols", [(), (0,)])
def test_sdc_search_matches_oracle(B, cluster_cols):
    say(f"[sdc] search cols={cluster_cols}")
    w = make_workload("c1", device="cuda", n_queries=24)
    idx = B.Index.from_workload(w, max_batch=24, max_k=w.k, cluster_cols=cluster_cols)
    ox = oracle_index(w.codes, w.C_pq, w.attrs)
    T = O.sdc_table(ox["C_pq"])
    preds = w.preds[w.bins[0]][:24]
    preds = preds[:20] + [[], [(0, 5, 5)], [(0, 0, 1000)], [(0, 17, 18)]]
    lut = idx.build_sdc_lut(w.queries)
    ids, dist = idx.search(preds, lut, w.k)
    torch.cuda.synchronize()
    ids, dist = _np(ids), _np(dist)
    for i, p in enumerate(preds):
        res = O.sdc_filtered_search(ox, _np(w.queries[i]), p, w.k, table=T)
        check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"sdc q{i} {p}")


def test_sdc_query_at_a_row_finds_it_first(B):
    """A query equal to row v's reconstruction has SDC distance 0 to v (and
    to rows with the same codes, which precede or follow by id)."""
    ix = random_index(20_000, 48, 2, 1, 5, 77, device="cuda")
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=8, max_k=10, cluster_cols=(0,))
    rows = [3, 999, 12_345, 19_999]
    q = torch.stack([ix["C_pq"][torch.arange(48, device="cuda"), ix["codes"][v].long()].reshape(-1) for v in rows])
    lut = idx.build_sdc_lut(q)
    ids, dist = idx.search([[]] * len(rows), lut, 10)
    torch.cuda.synchronize()
    for i, v in enumerate(rows):
        assert _np(dist[i])[0] == 0.0 and _np(ids[i])[0] == v
