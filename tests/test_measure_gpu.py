"""Measurement builds on the GPU: the read-counting build of the scan answers
exactly as the timed scan and counts every table read it issues; the LDS
gather probe reports rates in the range a 256-CU chip can reach."""
import numpy as np
import pytest
import torch

import oracle as O
from workload import random_index
from tests._gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


def _case(B, N=20_037, M=48, nq=40):
    ix = random_index(N, M, 2, 1, 1000, seed=91, device="cuda")
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=64, max_k=10, cluster_cols=(0,))
    g = torch.Generator(device="cpu").manual_seed(5)
    q = torch.randn(nq, M * 2, generator=g).cuda()
    preds = []
    for i in range(nq):
        lo = int(torch.randint(0, 1000, (1,), generator=g))
        w = [0, 1, 7, 50, 300, 1000][i % 6]
        preds.append([(0, lo, lo + w)])
    n_sel = sum(int(O.predicate_mask(ix["attrs"].cpu().numpy(), p).sum()) for p in preds)
    return ix, idx, q, preds, n_sel


def _interval_tiles(ix, preds):
    """64-row tiles of the clustered layout (rows sorted by the attribute)
    that hold a row of each query's interval, summed over the queries."""
    a = np.sort(ix["attrs"][0].cpu().numpy())
    tiles = 0
    for p in preds:
        (_, lo, hi), = p
        r0, r1 = int(np.searchsorted(a, lo)), int(np.searchsorted(a, hi))
        if r1 > r0:
            tiles += (r1 - 1) // 64 - r0 // 64 + 1
    return tiles


def _counted(B, idx, preds, lut):
    idx.set_option(B.OPT_COUNT_READS, 1)
    idx.read_scan_reads()
    ids, dist = idx.search(preds, lut, 10)
    hist = idx.read_scan_reads()
    idx.set_option(B.OPT_COUNT_READS, 0)
    return ids, dist, hist


def test_counting_scan_same_results_and_every_read_counted(B):
    say("[measure] counting build, no early abandonment")
    ix, idx, q, preds, n_sel = _case(B)
    M = ix["codes"].shape[1]
    lut = idx.build_lut(q, None, None, B.LUT_F32)
    # A negative entry in every table: partial sums no longer bound the full
    # sum, so no lane drops out and every selected row costs M reads.
    lut[:, 0, 0] = -1.0
    ids0, d0 = idx.search(preds, lut, 10)
    ids1, d1, hist = _counted(B, idx, preds, lut)
    torch.cuda.synchronize()
    assert torch.equal(ids0, ids1) and torch.equal(d0.view(torch.int32), d1.view(torch.int32))
    assert hist[0] == _interval_tiles(ix, preds)    # entry 0: every tile of each interval, once
    assert sum(n * hist[n] for n in range(1, 65)) == M * n_sel
    assert sum(hist[1:65]) % 8 == 0    # reads come in groups of 8 subspaces at M = 48


def test_counting_scan_with_early_abandonment(B):
    say("[measure] counting build, early abandonment")
    ix, idx, q, preds, n_sel = _case(B)
    M = ix["codes"].shape[1]
    lut = idx.build_lut(q, None, None, B.LUT_F32)
    ids0, d0 = idx.search(preds, lut, 10)
    ids1, d1, hist = _counted(B, idx, preds, lut)
    torch.cuda.synchronize()
    assert torch.equal(ids0, ids1) and torch.equal(d0.view(torch.int32), d1.view(torch.int32))
    lookups = sum(n * hist[n] for n in range(1, 65))
    assert hist[0] == _interval_tiles(ix, preds)
    # the first group of 8 subspaces is read for every selected row, the rest
    # only while a row can still enter the top k
    assert 8 * n_sel <= lookups <= M * n_sel
    assert lookups < M * n_sel


def test_counting_rejects_plans_without_a_counting_build(B):
    ix = random_index(5000, 12, 2, 1, 100, seed=3, device="cuda")   # M = 12: generic-M scan
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=8, max_k=10, cluster_cols=(0,))
    lut = idx.build_lut(torch.randn(4, 24, device="cuda"), None, None, B.LUT_F32)
    idx.set_option(B.OPT_COUNT_READS, 1)
    with pytest.raises(B.IfvsError):
        idx.search([[(0, 0, 50)]] * 4, lut, 5)
    idx.set_option(B.OPT_COUNT_READS, 0)
    ids, _ = idx.search([[(0, 0, 50)]] * 4, lut, 5)
    assert ids.shape == (4, 5)


def test_lds_gather_probe_rates(B):
    say("[measure] LDS gather probe")
    full = B.probe_lds_gather(64)
    half = B.probe_lds_gather(32)
    one = B.probe_lds_gather(1)
    cus, clk = 256, 2.4e9
    # a random 64-lane read takes between 2 (no conflicts) and 64 cycles of a CU's LDS
    assert cus * clk / 64 <= full <= cus * clk / 2 * 1.05, full
    # fewer lanes never make an instruction slower
    assert half >= 0.95 * full and one >= 0.95 * half, (full, half, one)
    for bad in (0, 65):
        with pytest.raises(B.IfvsError):
            B.probe_lds_gather(bad)
