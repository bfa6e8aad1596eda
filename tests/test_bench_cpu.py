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


def test_union_bytes_count_each_selected_tile_once():
    class W:
        M, N = 48, 6400
    sorted_attr = torch.arange(6400) // 10            # value v on rows [10v, 10v + 10)
    preds = [[(0, 0, 10)], [(0, 5, 20)], [(0, 100, 101)], [(0, 3, 3)]]
    # rows [0, 100), [50, 200), [1000, 1010), none: tiles [0, 2) + [0, 4) + [15, 16) -> 5 tiles
    got = bench.scan_union_bytes(W, sorted_attr, preds, {"splits": 2, "grid_tiles": 0}, 10, 4)
    assert got == 5 * 64 * 12 * 4 + 4 * 48 * 256 * 4 + 4 * 2 * bench.SCAN_WAVES * 10 * 8


def test_lds_roof_weights_reads_by_their_rate():
    hist = [0] * 65
    hist[64], hist[8] = 10, 4
    rate = [0.0] + [1e9] * 64
    rate[8] = 4e9
    lookups, secs = bench.lds_roof(hist, rate)
    assert lookups == 64 * 10 + 8 * 4
    assert abs(secs - (10 / 1e9 + 4 / 4e9)) < 1e-18
