"""Helpers shared by the GPU parity tests (not collected: no test_ prefix)."""
import sys

import numpy as np
import torch

import oracle as O


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def oracle_index(codes, C_pq, attrs, bank=None, W=None, r=0, h=0, hash_seed=0):
    c = lambda t: None if t is None else t.detach().cpu().numpy()
    return dict(codes=c(codes), C_pq=c(C_pq), attrs=c(attrs), bank=c(bank), W=c(W),
                r=int(r), h=int(h), hash_seed=int(hash_seed))


def oracle_from_workload(w, conditioned=True):
    return oracle_index(w.codes, w.C_pq, w.attrs, w.bank if conditioned else None,
                        w.W if conditioned else None, w.r, w.h, w.hash_seed)


def bits(a):
    a = np.ascontiguousarray(a)
    return a.view(np.uint32) if a.dtype == np.float32 else a.view(np.uint16)


def assert_bitexact(gpu, ref, what):
    g, r = bits(gpu), bits(ref)
    if not np.array_equal(g, r):
        bad = np.flatnonzero(g.ravel() != r.ravel())
        i = bad[0]
        raise AssertionError(f"{what}: {bad.size} of {g.size} differ; first at {i}: "
                             f"gpu={gpu.ravel()[i]!r} ref={ref.ravel()[i]!r}")


def check_search_row(ids_g, dist_g, ids_o, dist_o, what, dist64=None, rtol=1e-4):
    """ids bit-exact, distances bit-exact against the fp32 oracle, and within
    rtol of the fp64 definition where given."""
    if not np.array_equal(ids_g, ids_o):
        raise AssertionError(f"{what}: ids differ\n gpu={ids_g}\n ref={ids_o}")
    assert_bitexact(dist_g.astype(np.float32), dist_o.astype(np.float32), what + " dist")
    if dist64 is not None:
        fin = np.isfinite(dist64)
        assert np.all(np.isinf(dist_g[~fin]))
        err = np.abs(dist_g[fin].astype(np.float64) - dist64[fin])
        assert np.all(err <= rtol * np.maximum(np.abs(dist64[fin]), 1e-30)), (what, err.max())
