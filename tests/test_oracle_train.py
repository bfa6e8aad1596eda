"""Pins of the training oracle (one SGD step of the conditioning, Section 2,
training paragraph): its analytic gradients against central finite
differences of its forward loss, a two-candidate loss against the closed form
computed by hand, and the special cases the chain rule must respect."""
import math

import numpy as np
import pytest

from oracle import ifvs_train_oracle as T

K = 256


def _problem(seed, M=2, d=2, r=2, B=8, N=60, nq=3, n_cand=6, n_pos=2, wz=True):
    rng = np.random.default_rng(seed)
    C_pq = rng.normal(0, 1, (M, K, d))
    W = rng.normal(0, 0.3, (M, r, K, d))
    bank = rng.normal(0, 0.3, (B, M * r))
    codes = rng.integers(0, K, (N, M)).astype(np.uint8)
    # candidates drawn from few codewords so the table gradients pile up
    codes[:, 0] = codes[:, 0] % 5
    qs = rng.normal(0, 1, (nq, M * d)).astype(np.float32)
    preds = [[(0, i, i + 3)] for i in range(nq)]
    w_zs = rng.normal(0.5, 0.5, (nq, M * d)) if wz else None
    cands = np.stack([rng.choice(N, n_cand, replace=False) for _ in range(nq)]).astype(np.int64)
    return dict(qs=qs, preds=preds, w_zs=w_zs, cands=cands, n_pos=n_pos, bank=bank, W=W, C_pq=C_pq,
                codes=codes, h=2, hash_seed=7, tau=0.7, lam=0.3)


def _loss(p):
    return T.batch_loss(p["qs"], p["preds"], p["w_zs"], p["cands"], p["n_pos"], p["bank"], p["W"],
                        p["C_pq"], p["codes"], p["h"], p["hash_seed"], p["tau"], p["lam"])


def _grads(p):
    return T.batch_grads(p["qs"], p["preds"], p["w_zs"], p["cands"], p["n_pos"], p["bank"], p["W"],
                         p["C_pq"], p["codes"], p["h"], p["hash_seed"], p["tau"], p["lam"])


def _fd(p, key, idx, eps=1e-6):
    arr = p[key]
    old = arr[idx]
    arr[idx] = old + eps
    lp = _loss(p)
    arr[idx] = old - eps
    lm = _loss(p)
    arr[idx] = old
    return (lp - lm) / (2 * eps)


@pytest.mark.parametrize("seed", [1, 2])
def test_gradients_match_central_differences(seed):
    p = _problem(seed)
    g = _grads(p)
    rng = np.random.default_rng(100 + seed)
    touched = np.flatnonzero(np.abs(g["bank"]).sum(axis=1) > 0)
    assert touched.size > 0
    for row in touched:
        for col in range(p["bank"].shape[1]):
            fd = _fd(p, "bank", (row, col))
            assert abs(fd - g["bank"][row, col]) <= 1e-6 * max(1.0, abs(fd)), ("bank", row, col)
    # W entries on the codewords the candidates use, and random ones
    picks = [(m, t, int(p["codes"][p["cands"][0][0]][m]), j) for m in range(2) for t in range(2) for j in range(2)]
    picks += [tuple(int(rng.integers(0, s)) for s in p["W"].shape) for _ in range(24)]
    for idx in picks:
        fd = _fd(p, "W", idx)
        assert abs(fd - g["W"][idx]) <= 1e-6 * max(1.0, abs(fd)), ("W", idx)
    for i in range(len(p["qs"])):
        for j in range(p["w_zs"].shape[1]):
            fd = _fd(p, "w_zs", (i, j))
            assert abs(fd - g["w_z"][i, j]) <= 1e-6 * max(1.0, abs(fd)), ("w_z", i, j)
    # the per-query losses average to the batch loss
    assert math.isclose(g["loss"].mean(), _loss(p), rel_tol=1e-12)


def test_gradients_with_absent_candidates_and_unit_weights():
    p = _problem(3, wz=False, n_cand=7, n_pos=3)
    p["cands"][0, 1] = -1          # an absent positive
    p["cands"][1, 5] = -1          # an absent negative
    p["cands"][2, :3] = -1         # no positive: cross-entropy 0, anchor only
    g = _grads(p)
    assert g["w_z"] is None
    f = T.query_forward(p["qs"][2], p["preds"][2], None, p["cands"][2], 3, p["bank"], p["W"], p["C_pq"],
                        p["codes"], 2, 7, p["tau"], p["lam"])
    assert f["ce"] == 0.0 and f["reg"] > 0
    for idx in [(0, 0, 1, 0), (1, 1, 3, 1), (0, 1, int(p["codes"][p["cands"][0][0]][0]), 1)]:
        fd = _fd(p, "W", idx)
        assert abs(fd - g["W"][idx]) <= 1e-6 * max(1.0, abs(fd)), idx
    for row in np.flatnonzero(np.abs(g["bank"]).sum(axis=1) > 0):
        fd = _fd(p, "bank", (row, 2))
        assert abs(fd - g["bank"][row, 2]) <= 1e-6 * max(1.0, abs(fd)), row


def test_two_candidates_closed_form():
    """M = 1, d = 2, W = 0 (so C_iFVS = C_PQ), w_f = 1, q = 0: the positive's
    codeword is (1, 1), distance 2; the negative's is (1, 2), distance 5.
    With tau = 0.5 the loss is log(1 + e^{(2 - 5) / 0.5}) = log(1 + e^-6)."""
    C_pq = np.zeros((1, K, 2))
    C_pq[0, 3] = (1.0, 1.0)
    C_pq[0, 7] = (1.0, 2.0)
    codes = np.array([[7], [3]], dtype=np.uint8)
    f = T.query_forward(np.zeros(2, np.float32), [], None, [1, 0], 1, np.zeros((4, 2)), np.zeros((1, 2, K, 2)),
                        C_pq, codes, 2, 0, 0.5, 1.0)
    assert f["dist"].tolist() == [2.0, 5.0]
    assert f["reg"] == 0.0
    assert math.isclose(f["loss"], math.log1p(math.exp(-6.0)), rel_tol=1e-12)
    # one candidate (the positive alone): its cross-entropy is exactly 0
    f1 = T.query_forward(np.zeros(2, np.float32), [], None, [1], 1, np.zeros((4, 2)), np.zeros((1, 2, K, 2)),
                         C_pq, codes, 2, 0, 0.5, 1.0)
    assert f1["loss"] == 0.0


def test_zero_bank_leaves_W_untouched():
    """alpha = 0 (the initialization of the training paragraph): Delta = 0, and
    every W gradient is a multiple of alpha."""
    p = _problem(4)
    p["bank"][:] = 0.0
    g = _grads(p)
    assert np.all(g["W"] == 0.0)
    assert np.any(g["bank"] != 0.0)


def test_zero_W_leaves_bank_untouched():
    p = _problem(5)
    p["W"][:] = 0.0
    g = _grads(p)
    assert np.all(g["bank"] == 0.0)
    assert np.any(g["W"] != 0.0)


def test_equal_positive_distances_give_no_ranking_gradient():
    """Every candidate a positive, all on the same codes: the softmax equals
    the positives' share, so only the anchor term is left."""
    p = _problem(6, n_cand=4, n_pos=4)
    p["cands"] = np.arange(12, dtype=np.int64).reshape(3, 4)       # disjoint lists
    for i in range(len(p["qs"])):
        p["codes"][p["cands"][i]] = p["codes"][p["cands"][i][0]]
    lam = p["lam"]
    g = _grads(p)
    p["lam"] = 0.0
    g0 = _grads(p)
    assert np.allclose(g0["bank"], 0.0, atol=1e-15) and np.allclose(g0["W"], 0.0, atol=1e-15)
    assert np.allclose(g0["w_z"], 0.0, atol=1e-15)
    p["lam"] = 2 * lam
    g2 = _grads(p)
    assert np.allclose(g2["W"], 2 * g["W"], rtol=1e-12, atol=1e-15)   # anchor gradient linear in lam


def test_sgd_step_decreases_the_loss():
    p = _problem(7)
    l0 = _loss(p)
    g = _grads(p)
    p["bank"] = p["bank"] - 0.05 * g["bank"]
    p["W"] = p["W"] - 0.05 * g["W"]
    assert _loss(p) < l0
