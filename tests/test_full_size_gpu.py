"""Full-size workloads on the GPU, checked against the oracle.

Every returned row of a batch is checked for properties that hold at any
size (ids pass the predicate, ascending (distance, id), no duplicates, count
= min(k, |P|), identical on both row layouts), and the oracle recomputes
whole query sets one by one, in a pool of host processes, for an
element-by-element comparison of ids and distance bits:

* 10M x 96 (c4), in the launch configuration the benchmark times (clustered
  rows, conditioned mode, batches of 256, k = 10, fp32 tables, coarse
  quantizer of 2048 centroids: the list scan in the 10% and 50% bins): all
  256 queries of a batch in each of the four bins;
* 1M x 128 with a range and a category clause (c2): 64 queries per bin;
* 1M x 960 with k = 100 (c3): 32 queries per bin, and 8 more in the fp16
  table mode;
* 100M x 128 (c5): 16 queries per bin.

The counts can be raised with IFVS_FULL_ORACLE_SCALE (a multiplier, capped
at each batch's size)."""
import os

import numpy as np
import pytest
import torch

from oracle.pool import OraclePool, host_cores
from workload import make_workload
from tests._gpu_util import check_search_row, oracle_from_workload, say

pytestmark = pytest.mark.gpu

SCALE = float(os.environ.get("IFVS_FULL_ORACLE_SCALE", "1"))


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


def _workers():
    # the machine's CPU share, leaving one core to the test process
    return max(1, min(15, host_cores() - 1))


def _run_config(B, w, idx, plain, bins, nq, k, per_bin, conditioned=True, lut_dtype="f32", list_bins=()):
    """Searches the first nq queries of every bin on the GPU, checks the
    properties of every row, and compares the first per_bin[s] queries of
    bin s with the oracle.  With a coarse build on idx, the bounded search
    runs too (it must take the list scan in list_bins) and must return the
    same ids and distance bits."""
    dt = B.LUT_F16 if lut_dtype == "f16" else B.LUT_F32
    tasks, got = [], {}
    for s in bins:
        say(f"[full] {w.name} N={w.N} bin={s} ({lut_dtype})")
        preds = w.preds[s][:nq]
        q, wz = w.queries[:nq], w.w_z[s][:nq]
        a, f = idx.select_codebook(q, preds, wz)
        lut = idx.build_lut(q, a if conditioned else None, f, dt)
        ids, dist = idx.search(preds, lut, k, dt)
        _, counts = idx.filter(preds)
        torch.cuda.synchronize()
        _properties(w, preds, ids, dist, counts, k)
        if list_bins:
            ib, db = idx.search_bounded(preds, lut, a if conditioned else None, f, k, dt)
            torch.cuda.synchronize()
            assert idx.last_coarse() == (s in list_bins), (s, idx.last_coarse())
            assert torch.equal(ids, ib) and torch.equal(dist.view(torch.int32), db.view(torch.int32)), s
        if plain is not None:
            i2, d2 = plain.search(preds, lut, k, dt)
            torch.cuda.synchronize()
            assert torch.equal(ids, i2) and torch.equal(dist.view(torch.int32), d2.view(torch.int32))
        ids_h, dist_h, q_h, wz_h = _np(ids), _np(dist), _np(q), _np(wz)
        n_or = min(nq, int(round(per_bin[s] * SCALE)))
        for i in range(n_or):
            key = (s, i)
            got[key] = (ids_h[i], dist_h[i])
            tasks.append((key, q_h[i], preds[i], k, wz_h[i], lut_dtype, conditioned))
    ox = oracle_from_workload(w, conditioned)
    last = [0]

    def progress(done, total):
        if done == total or done - last[0] >= max(1, total // 10):
            last[0] = done
            say(f"[full] {w.name}: oracle {done}/{total}")

    say(f"[full] {w.name}: {len(tasks)} queries to the oracle on {_workers()} host processes")
    with OraclePool(ox, _workers()) as pool:
        results = pool.search(tasks, progress)
    for key, ids_o, dist_o, *_ in results:
        g_ids, g_d = got[key]
        check_search_row(g_ids, g_d, ids_o, dist_o, f"{w.name} s={key[0]} q{key[1]} ({lut_dtype})")
    return len(results)


def test_c4_10m_bench_configuration(B):
    say("[full] generating c4 (10M x 96)")
    w = make_workload("c4", device="cuda", n_queries=256, keep_x=False)
    clus = B.Index.from_workload(w, max_batch=256, max_k=10, cluster_cols=(0,))
    plain = B.Index.from_workload(w, max_batch=256, max_k=10)
    say("[full] c4: coarse quantizer, 2048 centroids")
    clus.build_coarse(2048, 20)
    # the bench's path: the list scan with the coarse bound in the 10% and 50%
    # bins, equal to the interval scan's answers and so to the oracle's
    n = _run_config(B, w, clus, plain, w.bins, 256, 10, {s: 256 for s in w.bins}, list_bins=(0.1, 0.5))
    assert n == 4 * 256


def test_c2_1m_two_attributes(B):
    say("[full] generating c2 (1M x 128, two attributes)")
    w = make_workload("c2", device="cuda", n_queries=64, keep_x=False)
    clus = B.Index.from_workload(w, max_batch=64, max_k=10, cluster_cols=(1, 0))
    plain = B.Index.from_workload(w, max_batch=64, max_k=10)
    _run_config(B, w, clus, plain, w.bins, 64, 10, {s: 64 for s in w.bins})


def test_c3_1m_960d_k100(B):
    say("[full] generating c3 (1M x 960, M = 120, k = 100)")
    w = make_workload("c3", device="cuda", n_queries=32, keep_x=False)
    clus = B.Index.from_workload(w, max_batch=32, max_k=100, cluster_cols=(0,))
    _run_config(B, w, clus, None, w.bins, 32, 100, {s: 32 for s in w.bins})
    # the fp16 table mode on the same data
    _run_config(B, w, clus, None, [0.01], 8, 100, {0.01: 8}, lut_dtype="f16")


def test_c5_100m(B):
    say("[full] generating c5 (100M x 128, codes only)")
    w = make_workload("c5", device="cuda", n_queries=16, keep_x=False)
    clus = B.Index.from_workload(w, max_batch=16, max_k=10, cluster_cols=(1, 0))
    _run_config(B, w, clus, None, w.bins, 16, 10, {s: 16 for s in w.bins})
