"""ifvs_filtered_search_noalloc against ifvs_filtered_search: the same ids and
distance bits, call after call (the second call of each pair with a smaller
batch, on the static workspace the first one left behind), on the clustered
and the bitmap layouts, with chunk-grid scans, selection bitmaps returned,
and a batch too large for the static workspace rejected without writing."""
import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu_util import check_search_row, oracle_index, say
from workload import random_index

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


def _preds(rng, nq, domain, width, extra_col=False):
    out = []
    for _ in range(nq):
        lo = int(rng.integers(0, domain - width))
        p = [(0, lo, lo + width)]
        if extra_col:
            p.append((1, 0, int(rng.integers(5, 50))))
        out.append(p)
    return out


def _both(B, idx, preds, lut, k, want_bitmap=False):
    """(ids, dist, bitmap) of the allocating search and of the static one."""
    nq = len(preds)
    pc = B.pack_predicates(preds)
    res = []
    for fn in (idx.search_into, idx.search_noalloc_into):
        ids = torch.full((nq, k), -7, device="cuda", dtype=torch.int32)
        dist = torch.full((nq, k), -7.0, device="cuda")
        bm = torch.zeros(nq, idx.words(), device="cuda", dtype=torch.int32) if want_bitmap else None
        fn(nq, pc, lut, B.LUT_F32, k, ids, dist, bm)
        torch.cuda.synchronize()
        res.append((ids.cpu().numpy(), dist.cpu().numpy(), None if bm is None else bm.cpu().numpy()))
    return res


def _same(a, b, what):
    assert np.array_equal(a[0], b[0]), f"{what}: ids differ"
    assert np.array_equal(a[1].view(np.uint32), b[1].view(np.uint32)), f"{what}: distance bits differ"
    if a[2] is not None:
        assert np.array_equal(a[2], b[2]), f"{what}: bitmaps differ"


@pytest.mark.parametrize("layout", ["clustered", "bitmap"])
def test_noalloc_matches_search_twice_second_smaller(B, layout):
    say(f"[noalloc] {layout}")
    rng = np.random.default_rng(11)
    ix = random_index(300_000, 48, 2, 2, 3650, 21, device="cuda")
    cols = (0,) if layout == "clustered" else ()
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], ix["hash_seed"],
                  max_batch=96, max_k=32, cluster_cols=cols)
    ox = oracle_index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], ix["hash_seed"])
    g = torch.Generator(device="cuda").manual_seed(5)
    for call, (nq, width, k) in enumerate([(96, 365, 10), (17, 37, 32)]):
        preds = _preds(rng, nq, 3650, width, extra_col=(layout == "bitmap"))
        q = torch.randn(nq, 96, device="cuda", generator=g)
        wz = 0.5413 + 0.1 * torch.randn(nq, 96, device="cuda", generator=g)
        alpha, wf = idx.select_codebook(q, preds, wz)
        lut = idx.build_lut(q, alpha, wf)
        a, b = _both(B, idx, preds, lut, k, want_bitmap=(call == 1))
        _same(a, b, f"{layout} call {call} nq={nq}")
        for i in (0, nq - 1):          # and the oracle agrees on a sample
            res = O.filtered_search(ox, q[i].cpu().numpy(), preds[i], k, w_z=wz[i].cpu().numpy())
            check_search_row(b[0][i], b[1][i], res["ids"], res["dist"], f"{layout} call {call} q{i}")


def test_noalloc_chunk_grid_scan(B):
    """Spans of 8192+ tiles take the chunk grid with its dispatch order."""
    say("[noalloc] chunk grid")
    rng = np.random.default_rng(12)
    ix = random_index(1_200_000, 16, 8, 1, 1000, 22, device="cuda")
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=64, max_k=16, cluster_cols=(0,))
    g = torch.Generator(device="cuda").manual_seed(6)
    for call, (nq, width) in enumerate([(64, 500), (9, 450)]):
        preds = _preds(rng, nq, 1000, width)
        lut = idx.build_lut(torch.randn(nq, 128, device="cuda", generator=g))
        a, b = _both(B, idx, preds, lut, 10)
        assert idx.last_plan()["grid_tiles"] > 0
        _same(a, b, f"grid call {call} nq={nq}")


def test_noalloc_rejects_batch_beyond_static_workspace(B):
    """Selection words of 256 queries over 2.1M rows need 67 MB: the static
    search refuses the batch before enqueuing anything, and a smaller batch
    on the same index then runs."""
    say("[noalloc] too large")
    rng = np.random.default_rng(13)
    ix = random_index(2_100_000, 16, 8, 2, 1000, 23, device="cuda")
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=256, max_k=10)
    preds = _preds(rng, 256, 1000, 100, extra_col=True)
    lut = idx.build_lut(torch.randn(256, 128, device="cuda"))
    ids = torch.full((256, 10), -7, device="cuda", dtype=torch.int32)
    dist = torch.full((256, 10), -7.0, device="cuda")
    with pytest.raises(B.IfvsError) as err:
        idx.search_noalloc_into(256, B.pack_predicates(preds), lut, B.LUT_F32, 10, ids, dist)
    assert err.value.status == B.E_INVALID and "scratch" in str(err.value)
    torch.cuda.synchronize()
    assert bool((ids == -7).all()) and bool((dist == -7.0).all())
    a, b = _both(B, idx, preds[:24], lut[:24].contiguous(), 10)
    _same(a, b, "after the refusal")
