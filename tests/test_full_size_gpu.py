"""Full-size workloads on the GPU, checked by sampling.

Every returned row of a batch is checked for properties that hold at any
size (ids pass the predicate, ascending (distance, id), no duplicates, count
= min(k, |P|), identical on both row layouts); a few queries per selectivity
bin are recomputed by the CPU oracle one by one (ids and distance bits).
c4 (10M vectors) runs in the launch configuration bench.py times: clustered
rows, conditioned mode, batches of 256, k = 10, fp32 tables."""
import numpy as np
import pytest
import torch

import oracle as O
from workload import make_workload
from tests._gpu_util import check_search_row, oracle_from_workload, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


def _np(t):
    return t.detach().cpu().numpy()


def _properties(w, preds, ids, dist, counts, k):
    """Checks on every row: ids pass the predicate (evaluated on the GPU with
    plain torch ops), ascending order, no duplicates, padding."""
    attrs = w.attrs
    for i, p in enumerate(preds):
        row_ids, row_d = ids[i], dist[i]
        n = int(min(k, int(counts[i])))
        assert torch.all(row_ids[:n] >= 0) and torch.all(row_ids[n:] == -1), (i, p)
        assert torch.all(torch.isinf(row_d[n:]))
        got = row_ids[:n].long()
        assert torch.unique(got).numel() == n
        for col, lo, hi in p:
            v = attrs[col][got].long()
            assert torch.all((v >= lo) & (v < hi)), (i, p)
        d = row_d[:n]
        assert torch.all(d[1:] >= d[:-1])
        ties = d[1:] == d[:-1]
        assert torch.all(got[1:][ties] > got[:-1][ties])


def _run_config(B, w, idx, plain, bins, nq, k, sample, conditioned=True, lut_dtype="f32"):
    dt = B.LUT_F16 if lut_dtype == "f16" else B.LUT_F32
    ox = oracle_from_workload(w, conditioned)
    for s in bins:
        say(f"[full] {w.name} N={w.N} bin={s}")
        preds = w.preds[s][:nq]
        q, wz = w.queries[:nq], w.w_z[s][:nq]
        a, f = idx.select_codebook(q, preds, wz)
        lut = idx.build_lut(q, a if conditioned else None, f, dt)
        ids, dist = idx.search(preds, lut, k, dt)
        _, counts = idx.filter(preds)
        torch.cuda.synchronize()
        _properties(w, preds, ids, dist, counts, k)
        if plain is not None:
            i2, d2 = plain.search(preds, lut, k, dt)
            torch.cuda.synchronize()
            assert torch.equal(ids, i2) and torch.equal(dist.view(torch.int32), d2.view(torch.int32))
        ids_h, dist_h = _np(ids), _np(dist)
        for i in range(sample):
            res = O.filtered_search(ox, _np(q[i]), preds[i], k, w_z=_np(wz[i]), lut_dtype=lut_dtype,
                                    conditioned=conditioned)
            check_search_row(ids_h[i], dist_h[i], res["ids"], res["dist"], f"{w.name} s={s} q{i}")


def test_c4_10m_bench_configuration(B):
    say("[full] generating c4 (10M x 96)")
    w = make_workload("c4", device="cuda", n_queries=256, keep_x=False)
    clus = B.Index.from_workload(w, max_batch=256, max_k=10, cluster_cols=(0,))
    plain = B.Index.from_workload(w, max_batch=256, max_k=10)
    _run_config(B, w, clus, plain, w.bins, 256, 10, sample=2)


def test_c2_1m_two_attributes(B):
    say("[full] generating c2 (1M x 128, two attributes)")
    w = make_workload("c2", device="cuda", n_queries=64, keep_x=False)
    clus = B.Index.from_workload(w, max_batch=64, max_k=10, cluster_cols=(1, 0))
    plain = B.Index.from_workload(w, max_batch=64, max_k=10)
    _run_config(B, w, clus, plain, w.bins, 64, 10, sample=2)


def test_c3_1m_960d_k100(B):
    say("[full] generating c3 (1M x 960, M = 120, k = 100)")
    w = make_workload("c3", device="cuda", n_queries=32, keep_x=False)
    clus = B.Index.from_workload(w, max_batch=32, max_k=100, cluster_cols=(0,))
    _run_config(B, w, clus, None, w.bins, 32, 100, sample=2)
    # the fp16 table mode on the same data
    _run_config(B, w, clus, None, [0.01], 8, 100, sample=1, lut_dtype="f16")


def test_c5_100m(B):
    say("[full] generating c5 (100M x 128, codes only)")
    w = make_workload("c5", device="cuda", n_queries=16, keep_x=False)
    clus = B.Index.from_workload(w, max_batch=16, max_k=10, cluster_cols=(1, 0))
    _run_config(B, w, clus, None, w.bins, 16, 10, sample=1)
