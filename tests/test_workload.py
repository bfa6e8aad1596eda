"""Seeded synthetic inputs: determinism, value ranges, realized selectivity per
bin and the truncated Zipf attribute."""
import hashlib

import numpy as np
import pytest
import torch

import oracle as O
from workload import base_chunks, make_workload
from workload.synth import CONFIGS, make_attributes, make_predicates, zipf_probs


def _sha(t):
    return hashlib.sha256(t.contiguous().cpu().numpy().tobytes()).hexdigest()


def test_deterministic_by_seed():
    a = make_workload("c1", n_queries=20)
    b = make_workload("c1", n_queries=20)
    for f in ("codes", "C_pq", "attrs", "queries", "bank", "W"):
        assert _sha(getattr(a, f)) == _sha(getattr(b, f)), f
    assert a.preds == b.preds
    assert _sha(a.w_z[0.1]) == _sha(b.w_z[0.1])


def test_c1_shapes_and_ranges():
    w = make_workload("c1")
    assert w.codes.shape == (10_000, 16) and w.codes.dtype == torch.uint8
    assert w.C_pq.shape == (16, 256, 8)
    assert w.attrs.shape == (1, 10_000) and int(w.attrs.min()) >= 0 and int(w.attrs.max()) < 1000
    assert w.queries.shape == (100, 128)
    assert all(len(p) == 1 and p[0][2] - p[0][1] == 100 for p in w.preds[0.1])
    # every one of the 256 codewords is used in most subspaces (k-means did not collapse)
    used = [len(torch.unique(w.codes[:, m])) for m in range(16)]
    assert min(used) > 200
    # the codes are nearest-centroid codes: reconstruction beats a random code
    x, C = w.x, w.C_pq
    xs = x.reshape(-1, 16, 8)
    rec = C[torch.arange(16)[None, :], w.codes.long()]
    err = ((xs - rec) ** 2).sum((1, 2)).mean()
    rnd = C[torch.arange(16)[None, :], torch.randint(0, 256, w.codes.shape)]
    assert err < 0.5 * ((xs - rnd) ** 2).sum((1, 2)).mean()


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c5"])
def test_realized_selectivity_per_bin(name):
    cfg = CONFIGS[name]
    attrs = make_attributes(cfg, 200_000).numpy()
    for b_i, s in enumerate(cfg["bins"]):
        preds = make_predicates(cfg, s, 60, 1000 * cfg["idx"] + 3 + 10 * b_i)
        real = np.mean([O.predicate_mask(attrs, p).mean() for p in preds])
        # binomial noise of 60 queries x N rows, plus rounding of range widths
        tol = max(0.25 * s, 4 * np.sqrt(s / (60 * attrs.shape[1])))
        assert abs(real - s) < tol, (name, s, real)


def test_zipf_frequencies_and_rank_prefix_reading():
    p = zipf_probs(100)
    assert abs(float(p[0]) - 1 / sum((c + 1) ** -1.1 for c in range(100))) < 1e-12
    assert abs(float(p[0]) - 0.2338) < 5e-4
    attrs = make_attributes(CONFIGS["c2"], 200_000)
    counts = torch.bincount(attrs[1].long(), minlength=100).double() / attrs.shape[1]
    assert torch.max(torch.abs(counts - p)) < 0.01
    # 50% bin: no category is frequent enough, so the category clause is a
    # rank prefix [0, c) whose mass first reaches 0.5 (c = 5)
    preds = make_predicates(CONFIGS["c2"], 0.5, 3, 99)
    assert all(pp[1][1:] == (0, 5) for pp in preds)


def test_base_chunks_regenerate_the_workload_vectors():
    """The chunk stream used for ground truth is the stream the codes were
    encoded from, at any chunk size that make_workload used."""
    w = make_workload("c1", n_queries=4, chunk_rows=3000)
    parts = list(base_chunks("c1", chunk_rows=3000))
    assert [p for p, _ in parts] == [0, 3000, 6000, 9000]
    assert torch.equal(torch.cat([c for _, c in parts]), w.x)
