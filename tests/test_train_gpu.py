"""One training step of the conditioning on the GPU (ifvs_train_step)
against the fp64 training oracle: per-query losses, the applied bank and W
updates (the change divided by the learning rate is the gradient), and
dL/dw_z, element by element within fp32 tolerances, on plain and clustered layouts, with absent candidates,
duplicate hashed rows and queries without positives; then that the trained
parameters are what the search uses."""
import numpy as np
import pytest
import torch

import oracle as O
from oracle import ifvs_train_oracle as T
from workload import random_index
from tests._gpu_util import check_search_row, say

pytestmark = pytest.mark.gpu

# Learning rate of the parity steps: a power of two, so lr * g is exact, and
# large enough that the read-back difference (old - new parameter) carries
# the gradient's own fp32 precision rather than the parameters' last bits.
LR = 1024.0


@pytest.fixture(scope="module")
def B():
    from paper_2607_22922_amd import ifvs
    return ifvs


def _np(t):
    return t.detach().cpu().numpy()


def _close(got, want, what, rel=2e-4):
    """Element by element: |gpu - oracle| <= rtol |oracle| + atol with
    rtol = rel / 2 and atol = rel / 4 x the array's largest magnitude, and
    the largest error within rel x that magnitude.  The floor covers fp32
    cancellation: each entry sums up to a few thousand fp32 terms of both
    signs (softmax weights of positives and negatives, Delta gradients over
    queries), whose rounding errors reach n 2^-24 ~ 1e-4 of the terms'
    magnitudes -- the same order as the largest entries (observed: at most
    4e-5 of the largest magnitude, on entries that cancel to near zero)."""
    scale = max(float(np.abs(want).max()), 1e-30)
    err = np.abs(got.astype(np.float64) - want)
    bound = 0.5 * rel * np.abs(want) + 0.25 * rel * scale
    bad = err > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} of {bad.size} entries off; worst excess at "
                           f"{int(np.argmax(err - bound))}: err {float(err.ravel()[np.argmax(err - bound)]):.3e}, "
                           f"want {float(np.ravel(want)[np.argmax(err - bound)]):.3e}, scale {scale:.3e}")
    assert float(err.max()) <= rel * scale, f"{what}: max |gpu - oracle| = {float(err.max()):.3e}, scale {scale:.3e}"


def _problem(B, seed, M, dsub, cluster_cols, nq=12, n_cand=24, n_pos=4, bank_rows=32, with_wz=True, scale=20.0):
    N = 6000
    ix = random_index(N, M, dsub, 2, 40, seed, device="cuda", bank_rows=bank_rows)
    ix["W"] *= scale                     # scale 20: Delta of the order of the codebook spread
    ix["bank"] *= scale
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], ix["hash_seed"],
                  max_batch=nq, max_k=16, cluster_cols=cluster_cols)
    g = torch.Generator(device="cuda").manual_seed(seed + 1)
    q = torch.randn(nq, M * dsub, device="cuda", generator=g)
    w_z = (0.5 + 0.4 * torch.randn(nq, M * dsub, device="cuda", generator=g)) if with_wz else None
    cand = torch.randint(0, N, (nq, n_cand), device="cuda", generator=g, dtype=torch.int32)
    cand[0, 1] = -1                     # an absent positive
    cand[1, n_cand - 1] = -1            # an absent negative
    cand[2, :n_pos] = -1                # no positive: anchor term only
    cand[3, 5] = N + 7                  # out of range: absent
    preds = [[(0, i, i + 20)] for i in range(nq)]
    return idx, ix, q, w_z, cand, preds, n_pos


def _oracle(ix, q, w_z, cand, preds, n_pos, tau, lam):
    cands = _np(cand).astype(np.int64)
    cands[(cands < 0) | (cands >= ix["codes"].shape[0])] = -1
    return T.batch_grads(_np(q), preds, None if w_z is None else _np(w_z).astype(np.float64), cands, n_pos,
                         _np(ix["bank"]).astype(np.float64), _np(ix["W"]).astype(np.float64),
                         _np(ix["C_pq"]).astype(np.float64), _np(ix["codes"]), ix["h"], ix["hash_seed"], tau, lam)


@pytest.mark.parametrize("cluster_cols,M,dsub", [((), 16, 4), ((0,), 16, 4), ((0,), 48, 2), ((), 8, 16)])
def test_train_step_matches_oracle(B, cluster_cols, M, dsub):
    say(f"[train] cols={cluster_cols} M={M} dsub={dsub}")
    idx, ix, q, w_z, cand, preds, n_pos = _problem(B, 5 + M, M, dsub, cluster_cols)
    tau, lam = 0.8, 0.05
    ref = _oracle(ix, q, w_z, cand, preds, n_pos, tau, lam)
    bank0, W0 = idx.read_params()
    loss, dwz = idx.train_step(q, preds, w_z, cand, n_pos, tau, lam, LR, want_dwz=True)
    bank1, W1 = idx.read_params()
    torch.cuda.synchronize()
    _close(_np(loss), ref["loss"], "loss", rel=1e-4)
    _close(_np((bank0 - bank1) / LR), ref["bank"], "bank gradient")
    _close(_np((W0 - W1) / LR), ref["W"], "W gradient")
    _close(_np(dwz), ref["w_z"], "w_z gradient")
    assert float(loss[2]) > 0 and abs(float(loss[2]) - ref["loss"][2]) <= 1e-4 * ref["loss"][2]


def test_train_step_without_w_z_and_duplicate_rows(B):
    """A one-row bank: both hash functions pick row 0, which receives both
    alpha gradients."""
    idx, ix, q, w_z, cand, preds, n_pos = _problem(B, 71, 16, 4, (0,), bank_rows=1, with_wz=False)
    tau, lam = 0.5, 0.2
    ref = _oracle(ix, q, None, cand, preds, n_pos, tau, lam)
    bank0, W0 = idx.read_params()
    loss, _ = idx.train_step(q, preds, None, cand, n_pos, tau, lam, LR)
    bank1, W1 = idx.read_params()
    torch.cuda.synchronize()
    _close(_np(loss), ref["loss"], "loss", rel=1e-4)
    _close(_np((bank0 - bank1) / LR), ref["bank"], "bank gradient")
    _close(_np((W0 - W1) / LR), ref["W"], "W gradient")


def test_trained_parameters_drive_the_search(B):
    """After a few steps the search (conditioned tables) uses the updated bank
    and W: its results equal the oracle's with the read-back parameters, and
    the training loss went down."""
    idx, ix, q, w_z, cand, preds, n_pos = _problem(B, 9, 16, 4, (0,), n_cand=16, n_pos=2, scale=1.0)
    losses = []
    for _ in range(6):
        loss, _ = idx.train_step(q, preds, w_z, cand, n_pos, 8.0, 0.01, 0.05)
        losses.append(float(loss.mean()))
    assert np.all(np.isfinite(losses)) and losses[-1] < losses[0], losses
    bank, W = idx.read_params()
    alpha, wf = idx.select_codebook(q, preds, w_z)
    lut = idx.build_lut(q, alpha, wf)
    ids, dist = idx.search(preds, lut, 10)
    torch.cuda.synchronize()
    for i in range(4):
        res_alpha, res_wf = O.select_codebook(_np(q[i]), preds[i], _np(bank), ix["h"], ix["hash_seed"], _np(w_z[i]))
        lut_o = O.build_lut(_np(q[i]), res_alpha, res_wf, _np(ix["C_pq"]), _np(W), 16, ix["r"])
        cand_o = O.passing_ids(O.predicate_mask(_np(ix["attrs"]), preds[i]))
        ids_o, dist_o = O.select_topk(O.adc_distances(lut_o, _np(ix["codes"]), cand_o), cand_o, 10)
        check_search_row(_np(ids[i]), _np(dist[i]), ids_o, dist_o, f"trained q{i}")


def test_train_step_errors(B):
    from tests.test_abi_gpu import _status
    ix = random_index(500, 8, 4, 1, 10, 3, device="cuda")
    plain = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], max_batch=4, max_k=8)
    lib = B.lib()
    q = torch.zeros(2, 32, device="cuda")
    cand = torch.zeros(2, 4, dtype=torch.int32, device="cuda")
    loss = torch.empty(2, device="cuda")
    pk = B.pack_predicates([[], []])
    st, msg = _status(B, lib.ifvs_train_step, plain.handle, 2, q.data_ptr(), pk, None, cand.data_ptr(), 4, 1,
                      0.5, 0.0, 0.1, loss.data_ptr(), None, None)
    assert st == B.E_STATE, msg
    idx = B.Index(ix["codes"], ix["C_pq"], ix["attrs"], ix["bank"], ix["W"], ix["r"], ix["h"], ix["hash_seed"],
                  max_batch=4, max_k=8)
    for args in ((2, 0, 0, 0.5, 0.0, 0.1), (2, 4, 5, 0.5, 0.0, 0.1), (2, 4, 1, 0.0, 0.0, 0.1),
                 (2, 4, 1, 0.5, -1.0, 0.1), (2, 4, 1, float("nan"), 0.0, 0.1), (5, 4, 1, 0.5, 0.0, 0.1),
                 (2, 4, 1, 0.5, 0.0, float("inf"))):
        nq, n_cand, n_pos, tau, lam, lr = args
        st, msg = _status(B, lib.ifvs_train_step, idx.handle, nq, q.data_ptr(), B.pack_predicates([[]] * nq), None,
                          cand.data_ptr(), n_cand, n_pos, tau, lam, lr, loss.data_ptr(), None, None)
        assert st == B.E_INVALID, (args, msg)
    st, msg = _status(B, lib.ifvs_train_step, idx.handle, 2, q.data_ptr(), pk, None, cand.data_ptr(), 4, 1,
                      0.5, 0.0, 0.1, loss.data_ptr(), loss.data_ptr(), None)
    assert st == B.E_INVALID and "w_z" in msg, msg
    st, msg = _status(B, lib.ifvs_read_params, plain.handle, None, None, None)
    assert st == B.E_STATE, msg


def test_training_loop_runs_and_fits_its_queries(B):
    """The training loop end to end on the 10K-vector workload: the
    conditioned search equals plain PQ before training (alpha = 0), the loss
    falls, and recall on the training queries does not drop."""
    from paper_2607_22922_amd import train
    out = train.main(["--config", "c1", "--bin", "0.1", "--train-queries", "64", "--test-queries", "32",
                      "--batch", "32", "--epochs", "4", "--n-neg", "16"])
    assert out["recall@10_conditioned_before"] == out["recall@10_identity"]
    losses = out["loss_per_epoch"]
    assert all(np.isfinite(losses)) and losses[-1] < losses[0], losses
    assert out["recall@10_conditioned_after"]["train"] >= out["recall@10_conditioned_before"]["train"]


def test_train_step_is_deterministic(B):
    """Two identical steps from identical states give identical bits (every
    sum of the step has a fixed order): bank, W, losses and dL/dw_z, with
    rows shared by several queries (a 3-row bank)."""
    outs = []
    for _ in range(2):
        idx, ix, q, w_z, cand, preds, n_pos = _problem(B, 33, 16, 4, (0,), bank_rows=3)
        loss, dwz = idx.train_step(q, preds, w_z, cand, n_pos, 0.8, 0.05, 1.0, want_dwz=True)
        bank, W = idx.read_params()
        torch.cuda.synchronize()
        outs.append([_np(t).copy() for t in (loss, dwz, bank, W)])
    for a, b, name in zip(outs[0], outs[1], ("loss", "dL/dw_z", "bank", "W")):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), name
