"""C ABI contract on the GPU: status codes, error text, and that a call that
fails validation writes nothing."""
import ctypes
import os
import subprocess
import sys

import pytest
import torch

from workload import random_index
from tests._gpu_util import say

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


@pytest.fixture(scope="module")
def small(B):
    ix = random_index(3000, 16, 8, 2, 50, 5, device="cuda")
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"],
                  ix["hash_seed"], max_batch=8, max_k=20)
    q = torch.randn(4, 128, device="cuda")
    lut = idx.build_lut(q)
    torch.cuda.synchronize()
    return idx, q, lut


def _status(B, fn, *args):
    st = fn(*args)
    return st, B.lib().ifvs_last_error().decode()


def test_search_argument_errors_write_nothing(B, small):
    idx, q, lut = small
    lib = B.lib()
    ids = torch.full((4, 10), 1234, device="cuda", dtype=torch.int32)
    dist = torch.full((4, 10), 7.0, device="cuda")
    good = B.pack_predicates([[(0, 0, 10)]] * 4)
    cases = {
        "k=0": (4, good, lut.data_ptr(), 0, 0),
        "k>max_k": (4, good, lut.data_ptr(), 0, 21),
        "nq>max_batch": (9, B.pack_predicates([[(0, 0, 10)]] * 9), lut.data_ptr(), 0, 10),
        "bad dtype": (4, good, lut.data_ptr(), 7, 10),
        "null lut": (4, good, None, 0, 10),
        "misaligned lut": (4, good, lut.data_ptr() + 4, 0, 10),
        "column out of range": (4, B.pack_predicates([[(2, 0, 10)]] * 4), lut.data_ptr(), 0, 10),
        "negative column": (4, B.pack_predicates([[(-1, 0, 10)]] * 4), lut.data_ptr(), 0, 10),
        "5 clauses": (4, B.pack_predicates([[(0, 0, 10)] * 5] * 4), lut.data_ptr(), 0, 10),
    }
    for name, (nq, preds, lp, dt, k) in cases.items():
        st, msg = _status(B, lib.ifvs_filtered_search, idx.handle, nq, preds, lp, dt, k,
                          ids.data_ptr(), dist.data_ptr(), None, torch.cuda.current_stream().cuda_stream)
        assert st == B.E_INVALID, (name, st, msg)
        assert msg and msg != "no error", name
    torch.cuda.synchronize()
    assert torch.all(ids == 1234) and torch.all(dist == 7.0)
    # reserved fields must be zero
    bad = B.pack_predicates([[(0, 0, 10)]] * 4)
    bad[1].c[0].reserved = 3
    st, msg = _status(B, lib.ifvs_filtered_search, idx.handle, 4, bad, lut.data_ptr(), 0, 10,
                      ids.data_ptr(), dist.data_ptr(), None, None)
    assert st == B.E_INVALID and "reserved" in msg
    # empty clause (lo >= hi) is not an error
    st, _ = _status(B, lib.ifvs_filtered_search, idx.handle, 4, B.pack_predicates([[(0, 9, 3)]] * 4),
                    lut.data_ptr(), 0, 10, ids.data_ptr(), dist.data_ptr(), None, None)
    assert st == B.OK
    torch.cuda.synchronize()
    assert torch.all(ids == -1) and torch.all(torch.isinf(dist))


def test_other_calls_validate(B, small):
    idx, q, lut = small
    lib = B.lib()
    wf = torch.empty(4, 128, device="cuda")
    st, _ = _status(B, lib.ifvs_select_codebook, idx.handle, 4, q.data_ptr(),
                    B.pack_predicates([[]] * 4), None, None, wf.data_ptr(), None)
    assert st == B.E_INVALID                       # alpha_out NULL with a memory bank
    st, _ = _status(B, lib.ifvs_build_lut, idx.handle, 4, None, None, None, 0, lut.data_ptr(), None)
    assert st == B.E_INVALID
    st, _ = _status(B, lib.ifvs_filter, idx.handle, 4, B.pack_predicates([[]] * 4), None, None, None)
    assert st == B.E_INVALID
    st, _ = _status(B, lib.ifvs_set_option, idx.handle, 99, 1)
    assert st == B.E_INVALID
    st, _ = _status(B, lib.ifvs_set_option, idx.handle, B.OPT_QTILE, -1)
    assert st == B.E_INVALID
    for opt, bad in ((B.OPT_PROFILE, 4), (B.OPT_GATHER, 3), (B.OPT_GRID_TILES, -5), (B.OPT_SLOT_ORDER, 2),
                     (B.OPT_GRID_RELATIVE, 2), (B.OPT_SHARED_BOUND, 3)):
        st, msg = _status(B, lib.ifvs_set_option, idx.handle, opt, bad)
        assert st == B.E_INVALID, (opt, bad, msg)
    for opt, good in ((B.OPT_GATHER, 2), (B.OPT_GATHER, 0), (B.OPT_GRID_TILES, 0), (B.OPT_SLOT_ORDER, 1),
                      (B.OPT_SLOT_ORDER, 0), (B.OPT_SHARED_BOUND, 1), (B.OPT_SHARED_BOUND, 2),
                      (B.OPT_SHARED_BOUND, 0)):
        assert lib.ifvs_set_option(idx.handle, opt, good) == B.OK
    for fn, args in ((lib.ifvs_filtered_search, (None, 1, None, None, 0, 1, None, None, None, None)),
                     (lib.ifvs_build_lut, (None, 1, None, None, None, 0, None, None))):
        assert fn(*args) == B.E_STATE
    # nq = 0 is a no-op
    assert lib.ifvs_filtered_search(idx.handle, 0, None, None, 0, 10, None, None, None, None) == B.OK


def test_profile_modes(B, small):
    """IFVS_OPT_PROFILE 1 times every kernel launch, 2 only the scans', 3
    only the list scan's (none here: no coarse build)."""
    idx, q, lut = small
    preds = [[(0, 0, 10)]] * 4
    for mode, timed in ((1, {"condition", "lut", "filter", "scan", "merge"}), (2, {"scan"}), (3, set())):
        idx.set_option(B.OPT_PROFILE, mode)
        idx.read_profile()
        a, f = idx.select_codebook(q, preds, None)
        lt = idx.build_lut(q, a, f)
        idx.search(preds, lt, 10)
        prof = idx.read_profile()
        got = {st for st, (ms, n) in prof.items() if n > 0}
        assert got == timed, (mode, prof)
        assert all(ms >= 0.0 for ms, _ in prof.values())
    idx.set_option(B.OPT_PROFILE, 0)


def test_load_validation(B):
    lib = B.lib()
    ix = random_index(100, 16, 8, 1, 10, 1, device="cuda")
    d = B.IndexDesc()
    d.n, d.dim, d.m, d.ksub, d.n_attr = 100, 128, 16, 256, 1
    d.codes, d.codebook, d.attrs = ix["codes"].data_ptr(), ix["C_pq"].data_ptr(), ix["attrs"].data_ptr()
    d.mem_kind, d.max_batch, d.max_k = B.MEM_DEVICE, 4, 10
    h = ctypes.c_void_p()
    for field, value in (("ksub", 128), ("dim", 100), ("max_k", 0), ("max_k", 2000), ("n", 0),
                         ("n_cluster", 3), ("mem_kind", 5)):
        old = getattr(d, field)
        setattr(d, field, value)
        assert lib.ifvs_load_index(ctypes.byref(d), ctypes.byref(h)) == B.E_INVALID, field
        setattr(d, field, old)
    d.n_cluster = 1
    d.cluster_col[0] = 4
    assert lib.ifvs_load_index(ctypes.byref(d), ctypes.byref(h)) == B.E_INVALID
    d.cluster_col[0] = 0
    assert lib.ifvs_load_index(ctypes.byref(d), ctypes.byref(h)) == B.OK
    lib.ifvs_free_index(h)


def test_lds_budget_unsupported_in_fp32_ok_in_fp16(B):
    """M = 160: one fp32 table is 160 KB, beyond a workgroup's LDS with its
    pools; the fp16 table fits."""
    say("[abi] LDS budget")
    ix = random_index(2000, 160, 1, 1, 10, 2, device="cuda")
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=2, max_k=10)
    q = torch.randn(2, 160, device="cuda")
    lut32 = idx.build_lut(q, lut_dtype=B.LUT_F32)
    with pytest.raises(B.IfvsError) as e:
        idx.search([[]] * 2, lut32, 10, B.LUT_F32)
    assert e.value.status == B.E_UNSUPPORTED
    lut16 = idx.build_lut(q, lut_dtype=B.LUT_F16)
    ids, dist = idx.search([[]] * 2, lut16, 10, B.LUT_F16)
    torch.cuda.synchronize()
    assert (ids >= 0).all()


def test_forced_allocation_failures_fail_cleanly():
    """IFVS_FAIL_ALLOC=n: the n-th allocation fails, load returns
    IFVS_E_NOMEM and nothing leaks; a later load in the same process works."""
    code = r"""
import ctypes, sys, torch
sys.path.insert(0, %r)
from paper_2607_22922_amd import ifvs as B
from workload import random_index
ix = random_index(500, 16, 8, 1, 10, 3, device="cuda")
try:
    B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], 1,
            max_batch=4, max_k=10, cluster_cols=(0,))
    print("LOADED")
except B.IfvsError as e:
    print("STATUS", e.status)
idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=4, max_k=10)
print("SECOND_OK")
""" % ROOT
    for n in (1, 4, 9):
        env = dict(os.environ, IFVS_FAIL_ALLOC=str(n))
        p = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                           timeout=240)
        assert p.returncode == 0, p.stderr[-2000:]
        assert f"STATUS {-2}" in p.stdout and "SECOND_OK" in p.stdout, (n, p.stdout)
