"""Predicate encoder on the GPU (ifvs_load_encoder / ifvs_encode_predicates)
against the fp64 oracle, and stage-wise parity of the search it feeds.

Tolerance: the kernel computes in fp32 (matrix-core projections, fp32 layer
norms and softmax); at these widths (dot products of at most 256 terms,
layer norms over at most 128) its deviation from the exact value is a few
fp32 ulps of the partial sums, far inside |gpu - exact| <= 1e-4 (|exact| +
0.01) for every element of w_z (|w_z| is about 0.5 here)."""
import numpy as np
import pytest
import torch

import oracle as O
from workload import random_encoder, random_index
from tests._gpu_util import check_search_row, oracle_index, say

pytestmark = pytest.mark.gpu

RTOL, FLOOR = 1e-4, 1e-2


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


def _np_enc(enc):
    out = {k: (v.detach().cpu().numpy() if torch.is_tensor(v) else v) for k, v in enc.items() if k != "layers"}
    out["layers"] = [{k: v.detach().cpu().numpy() for k, v in p.items()} for p in enc["layers"]]
    return out


def _preds(rng, n, n_attr, domains):
    out = []
    for i in range(n):
        cl = []
        for _ in range(i % 5):
            c = int(rng.integers(0, n_attr))
            lo = int(rng.integers(-50, domains[c]))
            w = int(rng.integers(0, domains[c] // 2 + 2))
            kind = rng.integers(0, 6)
            if kind == 0:
                cl.append((c, -(1 << 62), lo))
            elif kind == 1:
                cl.append((c, lo, 1 << 62))
            elif kind == 2:
                cl.append((c, lo, lo))               # empty clause
            else:
                cl.append((c, lo, lo + w))
        out.append(cl)
    return out


def _check_close(got, ref, what):
    err = np.abs(got.astype(np.float64) - ref)
    bad = err > RTOL * (np.abs(ref) + FLOOR)
    assert not bad.any(), f"{what}: {bad.sum()} elements off; worst {err.max():.3e} at {np.argmax(err)}"


@pytest.mark.parametrize("n_attr,D,H,heads,layers,F,nq", [
    (1, 96, 64, 4, 2, 128, 256),      # the 10M-vector workload's shape, a full batch
    (2, 128, 64, 4, 2, 128, 37),      # two attribute columns, a ragged batch
    (1, 960, 128, 8, 1, 256, 9),      # widest supported encoder, 960 output dimensions
    (3, 40, 32, 2, 3, 48, 5),         # three layers, odd sizes
    (2, 16, 16, 16, 1, 16, 4),        # one-dimensional heads
])
def test_encoder_matches_oracle(B, n_attr, D, H, heads, layers, F, nq):
    say(f"[encoder] n_attr={n_attr} D={D} H={H} heads={heads} layers={layers} F={F} nq={nq}")
    domains = [1000, 100, 3650][:n_attr]
    dsub = 8 if D % 8 == 0 and D >= 64 else 4
    ix = random_index(4096, D // dsub, dsub, n_attr, 100, seed=D + H, device="cuda")
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=max(nq, 8), max_k=10)
    enc = random_encoder(n_attr, D, domains, seed=7 * H + layers, hidden=H, heads=heads, layers=layers, ffn=F)
    idx.load_encoder(enc)
    rng = np.random.default_rng(nq + D)
    preds = _preds(rng, nq, n_attr, domains)
    wz = idx.encode_predicates(preds)
    torch.cuda.synchronize()
    wz = wz.cpu().numpy()
    en = _np_enc(enc)
    worst = 0.0
    for i, p in enumerate(preds):
        ref = O.encode_predicate(p, en)
        _check_close(wz[i], ref, f"query {i} {p}")
        worst = max(worst, float(np.max(np.abs(wz[i] - ref) / (np.abs(ref) + FLOOR))))
    say(f"[encoder] worst |gpu - oracle| / (|oracle| + {FLOOR}) = {worst:.2e}")


def test_encoder_feeds_the_search_stagewise(B):
    """w_z from the encoder -> select_codebook -> table -> search on a
    clustered index; the oracle, given the same w_z, returns the same ids and
    distance bits."""
    say("[encoder] stage-wise search")
    M, dsub = 16, 4
    ix = random_index(30_000, M, dsub, 2, 200, seed=5, device="cuda", bank_rows=97)
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], ix["hash_seed"],
                  max_batch=32, max_k=10, cluster_cols=(0,))
    idx.load_encoder(random_encoder(2, M * dsub, [200, 200], seed=3))
    preds = [[(0, 10 * i, 10 * i + 25)] + ([(1, 0, 100)] if i % 2 else []) for i in range(20)]
    q = torch.randn(len(preds), M * dsub, device="cuda", generator=torch.Generator(device="cuda").manual_seed(2))
    wz = idx.encode_predicates(preds)
    alpha, wf = idx.select_codebook(q, preds, wz)
    lut = idx.build_lut(q, alpha, wf)
    ids, dist = idx.search(preds, lut, 10)
    torch.cuda.synchronize()
    ox = oracle_index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], ix["hash_seed"])
    ids, dist, wz_h, q_h = ids.cpu().numpy(), dist.cpu().numpy(), wz.cpu().numpy(), q.cpu().numpy()
    for i, p in enumerate(preds):
        res = O.filtered_search(ox, q_h[i], p, 10, w_z=wz_h[i])
        check_search_row(ids[i], dist[i], res["ids"], res["dist"], f"q{i} {p}")


def test_encoder_errors(B):
    ix = random_index(1000, 8, 2, 1, 50, seed=9, device="cuda")
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=8, max_k=10)
    wz = torch.empty(2, 16, device="cuda")
    with pytest.raises(B.IfvsError) as e:
        idx.encode_predicates_into(2, B.pack_predicates([[], []]), wz)
    assert e.value.status == B.E_STATE
    enc = random_encoder(1, 16, [50], seed=1, hidden=32, heads=4, layers=1, ffn=32)
    bad = dict(enc, heads=5)                                   # does not divide H
    with pytest.raises(B.IfvsError):
        idx.load_encoder(bad)
    wide = random_encoder(1, 16, [50], seed=1, hidden=144, heads=4, layers=1, ffn=32)
    with pytest.raises(B.IfvsError):
        idx.load_encoder(wide)
    idx.load_encoder(enc)
    with pytest.raises(B.IfvsError):
        idx.encode_predicates([[]] * 9)                        # beyond max_batch
    with pytest.raises(B.IfvsError):
        idx.encode_predicates([[(3, 0, 1)]])                   # no column 3
    out = idx.encode_predicates([[], [(0, 1, 2)]])
    torch.cuda.synchronize()
    assert out.shape == (2, 16) and torch.isfinite(out).all()
