"""The benchmark's measurement helpers on the CPU: the streamed exact
filtered kNN used as recall ground truth equals a brute force over the
stored raw vectors (numpy, fp64) on one- and two-attribute workloads."""
import numpy as np
import pytest
import torch

import bench
import oracle as O
from workload import make_workload


def _brute(x, attrs, q, clauses, k):
    d = ((x.astype(np.float64) - q.astype(np.float64)[None, :]) ** 2).sum(1)
    ok = O.predicate_mask(attrs, clauses)
    ids = np.flatnonzero(ok)
    order = np.lexsort((ids, d[ids]))[:k]
    out = np.full(k, -1, dtype=np.int64)
    out[:order.size] = ids[order]
    return out


@pytest.mark.parametrize("name,N", [("c1", None), ("c2", 30_000)])
def test_streamed_ground_truth_equals_brute_force(name, N):
    w = make_workload(name, N=N, n_queries=6, chunk_rows=1 << 20)
    x, attrs = w.x.numpy(), w.attrs.numpy()
    preds = {s: w.preds[s][:6] for s in w.bins}
    if name == "c1":
        preds["extra"] = [[], [(0, 5, 6)], [(0, 9, 3)], [(0, 0, 1000)], [(0, 10, 900)], [(0, 300, 301)]]
    gt = bench.exact_filtered_knn(name, w.N, w.attrs, w.queries[:6], preds, w.k)
    for s, p in preds.items():
        for i in range(6):
            ref = _brute(x, attrs, w.queries[i].numpy(), p[i], w.k)
            assert np.array_equal(gt[s][i].numpy(), ref), (name, s, i, p[i])


def test_clause_tensors_padding_admits_everything():
    col, lo, hi = bench.clause_tensors([[], [(1, 3, 4)], [(0, -5, 7), (1, 0, 2)]], "cpu")
    assert col.shape == (3, 2)
    assert lo[0, 0] < -(1 << 40) and hi[0, 0] > (1 << 40)
    assert (col[1, 0], lo[1, 0], hi[1, 0]) == (1, 3, 4)
    assert (col[2, 1], lo[2, 1], hi[2, 1]) == (1, 0, 2)
