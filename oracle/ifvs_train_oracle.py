"""Plain CPU oracle of one training step of the iFVS conditioning.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``; never by the product path.

Section 2, training paragraph: training starts from alpha = 0 and w_f = 1;
for each training query-predicate pair the model builds the current
conditioned codebook and weights, scores the ground-truth positives, mines
hard negatives (the best-scoring candidates of the pool that are not ground
truth), adds an anchor regularizer that keeps C_iFVS close to C_PQ, and lets
the gradients flow through alpha into the memory bank and into W (and w_f);
C_PQ and the codes stay fixed.  The forward pass is the one of Section 2's
first display and Rank stage (conditioned codebook, weighted distances).

Readings (the paper names no loss, weight or optimizer; all listed in the
design notes):

* score = -distance / tau; the loss of a query is the multi-positive softmax
  cross-entropy of its candidate list (P positives first, then the hard
  negatives; id -1 marks an absent candidate):
      L_q = (1/P) sum_{p < P} [ logsumexp_v(-d_v / tau) + d_p / tau ],
  0 when the query has no positive.
* anchor regularizer: R_q = lam * mean over (m, c, j) of Delta_q[m, c, j]^2.
* the batch loss is the mean over queries of L_q + R_q; plain SGD.
* w_z has no encoder here (the predicate Transformer is out of scope): it is
  an input, and the step returns dL/dw_z for a caller that has one.

Everything is fp64.  The gradients are the chain rule written out; they are
pinned against central finite differences of ``batch_loss`` and against
special cases in ``tests/test_oracle_train.py``.
"""
from __future__ import annotations

import numpy as np

from .ifvs_oracle import KSUB, fingerprint, hashed_rows

__all__ = ["query_forward", "batch_loss", "batch_grads"]


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def query_forward(q, clauses, w_z, cand, n_pos, bank, W, C_pq, codes, h, hash_seed, tau, lam):
    """Forward pass of one query (Section 2, first display and Rank stage).

    q: [D] fp32 (its bytes are fingerprinted); w_z: [D] or None; cand: [n]
    original ids, the first n_pos the positives, -1 = absent; bank: [B][M*r];
    W: [M][r][K][d]; C_pq: [M][K][d]; codes: [N][M].  Returns a dict with the
    loss terms and every intermediate the gradients need."""
    M, r = W.shape[0], W.shape[1]
    d = C_pq.shape[2]
    rows = hashed_rows(fingerprint(np.asarray(q, dtype=np.float32), clauses), h, bank.shape[0], hash_seed)
    alpha = np.zeros(M * r)
    for row in rows:
        alpha = alpha + bank[row].astype(np.float64)
    a = alpha.reshape(M, r)
    if w_z is None:
        w = np.ones(M * d)
    else:
        wz = np.asarray(w_z, dtype=np.float64)
        w = np.log1p(np.exp(wz))
    Wd = W.astype(np.float64)
    delta = np.einsum("mt,mtcj->mcj", a, Wd)
    C = C_pq.astype(np.float64) + delta
    e = np.asarray(q, dtype=np.float64).reshape(M, 1, d) - C            # [M][K][d]
    wm = w.reshape(M, 1, d)
    lut = (wm * e * e).sum(axis=2)                                    # [M][K]
    cand = np.asarray(cand, dtype=np.int64)
    valid = cand >= 0
    pos = valid.copy()
    pos[n_pos:] = False
    dist = np.zeros(cand.shape[0])
    for i in np.flatnonzero(valid):
        dist[i] = lut[np.arange(M), codes[cand[i]].astype(np.int64)].sum()
    ce = 0.0
    p = np.zeros(cand.shape[0])
    n_p = int(pos.sum())
    if n_p > 0:
        s = -dist[valid] / tau
        mx = s.max()
        lse = mx + np.log(np.exp(s - mx).sum())
        p[valid] = np.exp(s - lse)
        ce = float((lse + dist[pos] / tau).sum() / n_p)
    reg = lam * float((delta * delta).mean())
    return {"rows": rows, "alpha": alpha, "w": w, "delta": delta, "e": e, "lut": lut, "dist": dist,
            "valid": valid, "pos": pos, "n_pos": n_p, "p": p, "ce": ce, "reg": reg, "loss": ce + reg}


def batch_loss(qs, preds, w_zs, cands, n_pos, bank, W, C_pq, codes, h, hash_seed, tau, lam):
    """Mean over the batch of L_q + R_q."""
    tot = 0.0
    for i in range(len(qs)):
        f = query_forward(qs[i], preds[i], None if w_zs is None else w_zs[i], cands[i], n_pos,
                          bank, W, C_pq, codes, h, hash_seed, tau, lam)
        tot += f["loss"]
    return tot / len(qs)


def batch_grads(qs, preds, w_zs, cands, n_pos, bank, W, C_pq, codes, h, hash_seed, tau, lam):
    """Per-query losses and the gradients of the batch loss with respect to
    the memory bank, W and each query's w_z.

    Returns {"loss": [nq], "bank": [B][M*r], "W": [M][r][K][d],
    "w_z": [nq][D] or None}."""
    nq = len(qs)
    M, r, K, d = W.shape
    g_bank = np.zeros(bank.shape)
    g_W = np.zeros(W.shape)
    g_wz = None if w_zs is None else np.zeros((nq, M * d))
    losses = np.zeros(nq)
    for i in range(nq):
        w_z = None if w_zs is None else w_zs[i]
        f = query_forward(qs[i], preds[i], w_z, cands[i], n_pos, bank, W, C_pq, codes, h, hash_seed, tau, lam)
        losses[i] = f["loss"]
        # d(mean loss)/d(distance of candidate v): softmax minus the
        # positives' share, times -1/tau, over the batch size.
        g_dist = np.zeros(f["dist"].shape[0])
        if f["n_pos"] > 0:
            g_s = f["p"] - f["pos"] / f["n_pos"]
            g_dist = -g_s / tau / nq
        # The table entries each candidate read.
        g_lut = np.zeros((M, K))
        for v in np.flatnonzero(f["valid"]):
            c = codes[int(cands[i][v])].astype(np.int64)
            for m in range(M):
                g_lut[m, c[m]] += g_dist[v]
        # lut[m][c] = sum_j w e^2 with e = q - C_pq - Delta.
        wm = f["w"].reshape(M, 1, d)
        g_delta = g_lut[:, :, None] * (-2.0 * wm * f["e"])
        g_delta += (lam * 2.0 / (M * K * d) / nq) * f["delta"]
        a = f["alpha"].reshape(M, r)
        g_alpha = np.einsum("mcj,mtcj->mt", g_delta, W.astype(np.float64)).reshape(M * r)
        g_W += np.einsum("mcj,mt->mtcj", g_delta, a)
        for row in f["rows"]:
            g_bank[row] += g_alpha
        if g_wz is not None:
            g_w = (g_lut[:, :, None] * f["e"] * f["e"]).sum(axis=1).reshape(M * d)
            g_wz[i] = g_w * _sigmoid(np.asarray(w_z, dtype=np.float64))
    return {"loss": losses, "bank": g_bank, "W": g_W, "w_z": g_wz}
