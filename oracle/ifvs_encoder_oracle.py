"""Plain CPU oracle of the predicate encoder: f -> w_z.

TEST INFRASTRUCTURE ONLY: imported by ``tests/`` and ``bench.py``'s oracle
leg; never by the product path.

Section 2, opening paragraph: the relational predicate f is encoded by a
light-weight Transformer into a filter-aware weight vector w_z in R^D, which
reweighs the dimensions of the query and the database vectors by their
relevance to f (then w_f = softplus(w_z), first display).  The paper gives
no architecture, so this build takes the following reading (listed in the
design notes):

* tokens: a summary token (a learned vector ``cls``) followed by one token
  per clause (col, lo, hi), in the predicate's order.  A clause token is
  col_embed[col] + a * feat_w[0] + b * feat_w[1] + feat_b, where
  a = clip((lo - col_offset[col]) * col_scale[col], -1, 2) and b the same of
  hi: the bounds normalized to the column's domain ([0, 1) inside it),
  computed in fp64 and clipped, so an open bound (+-2^62) is -1 or 2.  No
  positional encoding: a conjunction does not depend on its clause order.
* ``layers`` pre-norm Transformer encoder layers over all tokens (no mask):
      Z = LN1(X);  Q, K, V = Z Wq + bq, Z Wk + bk, Z Wv + bv
      head h (of ``heads``, width dh = H / heads): A_h = softmax over keys of
      Q_h K_h^T / sqrt(dh);  X = X + concat_h(A_h V_h) Wo + bo
      X = X + relu(LN2(X) W1 + b1) W2 + b2
  LN(x) = (x - mean(x)) / sqrt(mean((x - mean(x))^2) + 1e-5) * g + b over the
  hidden width H.  Matrices map rows: y = x W + b, W stored [in][out].
* output: w_z = LN_f(X[summary]) W_out + b_out, in R^D.

All arithmetic is in ``dtype`` (fp64 by default; the paper fixes no
precision).  Pins in ``tests/test_oracle_encoder.py``: equality with a stack
of ``torch.nn.TransformerEncoderLayer`` (a library implementation of the
same layer) carrying the same weights, clause-order invariance, a
hand-computed two-token example, the one-token (empty predicate) closed form
and the feature clipping.
"""
from __future__ import annotations

import numpy as np

__all__ = ["LN_EPS", "clause_features", "encoder_tokens", "layer_norm", "encoder_layer", "encode_predicate"]

LN_EPS = 1e-5


def clause_features(clause, col_offset, col_scale):
    """(a, b): the clause's bounds normalized by its column's offset and
    scale, in fp64, clipped to [-1, 2]."""
    col, lo, hi = int(clause[0]), int(clause[1]), int(clause[2])
    off, sc = float(col_offset[col]), float(col_scale[col])
    a = min(max((float(lo) - off) * sc, -1.0), 2.0)
    b = min(max((float(hi) - off) * sc, -1.0), 2.0)
    return a, b


def encoder_tokens(clauses, enc, dtype=np.float64):
    """The token matrix [1 + len(clauses)][H]: the summary token, then one
    token per clause."""
    cls = np.asarray(enc["cls"], dtype=dtype)
    rows = [cls.copy()]
    fw = np.asarray(enc["feat_w"], dtype=dtype)
    fb = np.asarray(enc["feat_b"], dtype=dtype)
    ce = np.asarray(enc["col_embed"], dtype=dtype)
    for cl in clauses:
        a, b = clause_features(cl, enc["col_offset"], enc["col_scale"])
        a, b = dtype(a), dtype(b)
        rows.append(ce[int(cl[0])] + a * fw[0] + b * fw[1] + fb)
    return np.stack(rows).astype(dtype)


def layer_norm(x, g, b, dtype=np.float64):
    """Row-wise layer normalization over the last axis (biased variance)."""
    x = np.asarray(x, dtype=dtype)
    mu = x.mean(axis=-1, keepdims=True)
    d = x - mu
    var = (d * d).mean(axis=-1, keepdims=True)
    return d / np.sqrt(var + dtype(LN_EPS)) * np.asarray(g, dtype=dtype) + np.asarray(b, dtype=dtype)


def _softmax_rows(s):
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


def encoder_layer(X, p, heads, dtype=np.float64):
    """One pre-norm layer over the token matrix X [S][H] (all tokens attend
    to all)."""
    f = lambda k: np.asarray(p[k], dtype=dtype)
    S, H = X.shape
    dh = H // heads
    Z = layer_norm(X, p["ln1_g"], p["ln1_b"], dtype)
    Q = Z @ f("Wq") + f("bq")
    K = Z @ f("Wk") + f("bk")
    V = Z @ f("Wv") + f("bv")
    O = np.empty_like(Q)
    for h in range(heads):
        sl = slice(h * dh, (h + 1) * dh)
        A = _softmax_rows((Q[:, sl] @ K[:, sl].T) / np.sqrt(dtype(dh)))
        O[:, sl] = A @ V[:, sl]
    X = X + O @ f("Wo") + f("bo")
    Z = layer_norm(X, p["ln2_g"], p["ln2_b"], dtype)
    Hd = np.maximum(Z @ f("W1") + f("b1"), dtype(0))
    return X + Hd @ f("W2") + f("b2")


def encode_predicate(clauses, enc, dtype=np.float64):
    """w_z [D] of one predicate (a list of (col, lo, hi) clauses)."""
    X = encoder_tokens(clauses, enc, dtype)
    for p in enc["layers"]:
        X = encoder_layer(X, p, int(enc["heads"]), dtype)
    z = layer_norm(X[0], enc["lnf_g"], enc["lnf_b"], dtype)
    return z @ np.asarray(enc["out_w"], dtype=dtype) + np.asarray(enc["out_b"], dtype=dtype)
