"""Pins of the predicate-encoder oracle (oracle/ifvs_encoder_oracle.py) to
things other than itself:

* a stack of torch.nn.TransformerEncoderLayer (pre-norm, ReLU, no dropout) --
  a library implementation of the same layer -- carrying the same weights,
  followed by torch's layer_norm and a matrix product, gives the same w_z
  from the same tokens;
* a two-token example worked out by hand: with identity projections the
  two-token softmax reduces to a hyperbolic tangent;
* an empty predicate (the summary token alone) attends only to itself, so
  its w_z cannot depend on the query and key projections;
* a conjunction does not depend on its clause order;
* bound features: in-domain bounds map to [0, 1], open bounds clip to -1 and
  2, and the clause token is the column embedding plus the bound projection.
"""
import math

import numpy as np
import pytest
import torch

from oracle.ifvs_encoder_oracle import LN_EPS, clause_features, encode_predicate, encoder_tokens
from workload import random_encoder


def _np_enc(enc):
    out = {k: (v.detach().cpu().numpy() if torch.is_tensor(v) else v) for k, v in enc.items() if k != "layers"}
    out["layers"] = [{k: v.detach().cpu().numpy() for k, v in p.items()} for p in enc["layers"]]
    return out


@pytest.fixture(scope="module")
def enc():
    return _np_enc(random_encoder(3, 40, [1000, 100, 3650], seed=17, hidden=32, heads=4, layers=2, ffn=48))


def _torch_reference(tokens, enc):
    """The same encoder from torch.nn building blocks (fp64, CPU)."""
    H = tokens.shape[1]
    heads = int(enc["heads"])
    F = enc["layers"][0]["W1"].shape[1]
    x = torch.tensor(tokens, dtype=torch.float64)[None]          # [1][S][H]
    for p in enc["layers"]:
        lay = torch.nn.TransformerEncoderLayer(H, heads, dim_feedforward=F, dropout=0.0, activation="relu",
                                               layer_norm_eps=LN_EPS, batch_first=True, norm_first=True,
                                               dtype=torch.float64)
        t = lambda a: torch.tensor(np.asarray(a), dtype=torch.float64)
        with torch.no_grad():
            lay.self_attn.in_proj_weight.copy_(torch.cat([t(p["Wq"]).T, t(p["Wk"]).T, t(p["Wv"]).T]))
            lay.self_attn.in_proj_bias.copy_(torch.cat([t(p["bq"]), t(p["bk"]), t(p["bv"])]))
            lay.self_attn.out_proj.weight.copy_(t(p["Wo"]).T)
            lay.self_attn.out_proj.bias.copy_(t(p["bo"]))
            lay.linear1.weight.copy_(t(p["W1"]).T)
            lay.linear1.bias.copy_(t(p["b1"]))
            lay.linear2.weight.copy_(t(p["W2"]).T)
            lay.linear2.bias.copy_(t(p["b2"]))
            lay.norm1.weight.copy_(t(p["ln1_g"]))
            lay.norm1.bias.copy_(t(p["ln1_b"]))
            lay.norm2.weight.copy_(t(p["ln2_g"]))
            lay.norm2.bias.copy_(t(p["ln2_b"]))
        lay.eval()
        with torch.no_grad():
            x = lay(x)
    z = torch.nn.functional.layer_norm(x[0, 0], (H,), torch.tensor(enc["lnf_g"], dtype=torch.float64),
                                       torch.tensor(enc["lnf_b"], dtype=torch.float64), LN_EPS)
    return (z @ torch.tensor(enc["out_w"], dtype=torch.float64)
            + torch.tensor(enc["out_b"], dtype=torch.float64)).numpy()


@pytest.mark.parametrize("clauses", [[], [(0, 100, 400)], [(2, 10, 14), (1, 3, 4)],
                                     [(0, -(1 << 62), 500), (1, 0, 1), (2, 3000, 1 << 62), (0, 7, 7)]])
def test_matches_torch_transformer_encoder_layers(enc, clauses):
    tokens = encoder_tokens(clauses, enc)
    ref = _torch_reference(tokens, enc)
    got = encode_predicate(clauses, enc)
    assert got.shape == (40,)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


def test_two_token_softmax_by_hand():
    """H = 2, one head, one layer, identity projections, no feed-forward.
    Summary token [1, 0], clause token [0, 1].  LN of [1, 0] is [c, -c] with
    c = 0.5 / sqrt(0.25 + eps) (and [-c, c] for the clause), so the scores
    are +-2c^2 / sqrt(2) and the two-token softmax gives the summary token
    O = tanh(sqrt(2) c^2) [c, -c].  After the residual, [1 + ct, -ct] has
    final LN [e, -e] with e = h / sqrt(h^2 + eps), h = (1 + 2ct) / 2."""
    eye, zero2 = np.eye(2), np.zeros(2)
    layer = dict(ln1_g=np.ones(2), ln1_b=zero2, Wq=eye, Wk=eye, Wv=eye, bq=zero2, bk=zero2, bv=zero2,
                 Wo=eye, bo=zero2, ln2_g=np.ones(2), ln2_b=zero2, W1=np.zeros((2, 2)), b1=zero2,
                 W2=np.zeros((2, 2)), b2=zero2)
    enc = dict(heads=1, col_offset=np.zeros(1), col_scale=np.ones(1), col_embed=np.array([[0.0, 1.0]]),
               feat_w=np.zeros((2, 2)), feat_b=zero2, cls=np.array([1.0, 0.0]), layers=[layer],
               lnf_g=np.ones(2), lnf_b=zero2, out_w=np.array([[1.0], [0.0]]), out_b=np.zeros(1))
    eps = 1e-5
    c = 0.5 / math.sqrt(0.25 + eps)
    t = math.tanh(math.sqrt(2.0) * c * c)
    h = (1.0 + 2.0 * c * t) / 2.0
    e = h / math.sqrt(h * h + eps)
    got = encode_predicate([(0, 0, 1)], enc)
    assert got.shape == (1,)
    assert abs(got[0] - e) < 1e-14
    # one token alone attends to itself: O = V = [c, -c], X = [1 + c, -c]
    h1 = (1.0 + 2.0 * c) / 2.0
    assert abs(encode_predicate([], enc)[0] - h1 / math.sqrt(h1 * h1 + eps)) < 1e-14


def test_empty_predicate_ignores_query_and_key_projections(enc):
    other = {k: v for k, v in enc.items()}
    rng = np.random.default_rng(3)
    other["layers"] = [dict(p, Wq=rng.standard_normal(p["Wq"].shape), Wk=rng.standard_normal(p["Wk"].shape),
                            bq=rng.standard_normal(p["bq"].shape)) for p in enc["layers"]]
    np.testing.assert_allclose(encode_predicate([], other), encode_predicate([], enc), rtol=1e-13, atol=1e-14)
    assert not np.allclose(encode_predicate([(0, 5, 9)], other), encode_predicate([(0, 5, 9)], enc))


def test_clause_order_does_not_matter(enc):
    f = [(0, 100, 400), (1, 3, 4), (2, 0, 365)]
    base = encode_predicate(f, enc)
    for perm in ([2, 0, 1], [1, 2, 0], [0, 2, 1]):
        np.testing.assert_allclose(encode_predicate([f[i] for i in perm], enc), base, rtol=1e-12, atol=1e-13)
    assert not np.allclose(encode_predicate([(0, 100, 401), (1, 3, 4), (2, 0, 365)], enc), base)


def test_bound_features_and_clause_token(enc):
    off, sc = enc["col_offset"], enc["col_scale"]
    assert clause_features((0, 0, 1000), off, sc) == (0.0, 1.0)
    assert clause_features((2, 365, 730), off, sc) == pytest.approx((0.1, 0.2), rel=1e-15)
    assert clause_features((1, -(1 << 62), 1 << 62), off, sc) == (-1.0, 2.0)
    assert clause_features((1, 150, 120), off, sc) == (1.5, 1.2)
    tok = encoder_tokens([(2, 365, 730)], enc)
    assert tok.shape == (2, 32)
    np.testing.assert_array_equal(tok[0], enc["cls"])
    f64 = lambda a: np.asarray(a, dtype=np.float64)
    np.testing.assert_allclose(tok[1], f64(enc["col_embed"][2]) + 0.1 * f64(enc["feat_w"][0])
                               + 0.2 * f64(enc["feat_w"][1]) + f64(enc["feat_b"]), rtol=1e-14, atol=1e-14)
