"""Pins of the CPU oracle against facts that do not come from the oracle itself:
published hash test vectors, hand-written byte layouts, closed forms, textbook
special cases computed by library routines, the paper's own score formula,
and brute force on tiny inputs."""
import math
import os
import struct

import numpy as np
import pytest
from scipy.spatial.distance import cdist

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
U32 = 2.0 ** -24          # unit roundoff of fp32


def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [l.split() for l in f if l.strip() and not l.startswith("#")]


# ------------------------------------------------------------------ hashes
def test_fnv1a64_published_vectors():
    rows = _golden_lines("fnv1a64.txt")
    assert len(rows) == 3
    for text, hexval in rows:
        data = text.strip('"').encode("ascii")
        assert O.fnv1a64(data) == int(hexval, 16)


def test_splitmix64_published_sequence():
    (row,) = _golden_lines("splitmix64.txt")
    seed, expected = int(row[0]), [int(v) for v in row[1:]]
    gamma = 0x9E3779B97F4A7C15
    got = [O.splitmix64((seed + i * gamma) % (1 << 64)) for i in range(len(expected))]
    assert got == expected


def test_fingerprint_byte_layout_written_out():
    # q = [1.0, -2.0] as fp32 LE, one clause (col 1, lo 5, hi 9)
    q = np.array([1.0, -2.0], dtype=np.float32)
    expect = bytes.fromhex(
        "0000803f" "000000c0"                  # 1.0f, -2.0f
        "01000000"                             # one clause
        "01000000" "0500000000000000" "0900000000000000")
    assert O.fingerprint_bytes(q, [(1, 5, 9)]) == expect
    assert O.fingerprint(q, [(1, 5, 9)]) == O.fnv1a64(expect)
    # the empty predicate is the clause count 0 only
    assert O.fingerprint_bytes(q, []) == expect[:8] + bytes(4)


def test_hashed_rows_range_seed_and_spread():
    B = 64
    keys = [O.fnv1a64(struct.pack("<i", i)) for i in range(4000)]
    rows0 = np.array([O.hashed_rows(k, 2, B, 7) for k in keys])
    assert rows0.min() >= 0 and rows0.max() < B
    # two hash functions disagree for most keys, and a new seed changes rows
    assert np.mean(rows0[:, 0] != rows0[:, 1]) > 0.9
    rows1 = np.array([O.hashed_rows(k, 2, B, 8) for k in keys])
    assert np.mean(rows0 != rows1) > 0.9
    # roughly uniform: chi-square over 64 bins with 8000 draws
    counts = np.bincount(rows0.ravel(), minlength=B)
    exp = rows0.size / B
    chi2 = ((counts - exp) ** 2 / exp).sum()
    assert chi2 < 120          # 63 d.o.f.; p ~ 1e-5 at 120
    # definition written out for one key: row_i = sm(key ^ sm(seed + i)) mod B
    k = keys[5]
    assert O.hashed_rows(k, 1, B, 7)[0] == O.splitmix64(k ^ O.splitmix64(7)) % B


def test_hashed_row_from_published_splitmix64_outputs():
    """A bank row fixed by the published SplitMix64 sequence alone.  With seed
    s0 the generator's first two outputs are SM(s0) and SM(s0 + gamma).  Take
    hash function i = 3 under seed s0 + gamma - 3: its salt is
    SM(s0 + gamma), the second published output; for the key
    (second output) XOR s0, key XOR salt = s0, whose hash is the first
    published output.  So row_3 = (first output) mod B, an integer computed
    here without the oracle.  B = 45,000 is a bank size of the paper's
    Table 2 (not a power of two, so mod and a bit mask differ), 4,097 a
    second non-power-of-two check."""
    (row,) = _golden_lines("splitmix64.txt")
    s0, out1, out2 = int(row[0]), int(row[1]), int(row[2])
    gamma, mask = 0x9E3779B97F4A7C15, (1 << 64) - 1
    seed = (s0 + gamma - 3) & mask
    assert (seed ^ 3) != (seed + 3) & mask          # salting by seed XOR i would differ
    key = out2 ^ s0
    for B in (45000, 4097):
        rows = O.hashed_rows(key, 4, B, seed)
        assert rows[3] == out1 % B, (B, rows)
        assert all(0 <= r < B for r in rows)


def test_hashed_rows_seed_shift():
    """Hash function i under seed s is hash function 0 under seed s + i (the h
    functions are the members s, s + 1, ..., s + h - 1 of one family), for
    seeds where adding i carries across bits."""
    rng = np.random.default_rng(5)
    for t in range(200):
        key = int(rng.integers(0, 1 << 63)) * 2 + t % 2
        seed = int(rng.integers(0, 1 << 62)) | 0x7             # low bits set: s + i carries
        B = int(rng.integers(2, 100000))
        rows = O.hashed_rows(key, 6, B, seed)
        for i in range(6):
            assert rows[i] == O.hashed_rows(key, 1, B, seed + i)[0], (t, i)


@pytest.mark.parametrize("B", [45000, 4097])
def test_hashed_rows_cover_non_power_of_two_bank(B):
    """Rows reach every part of a bank whose size is not a power of two:
    close to all rows are hit and the hits are uniform over 45 (or 17)
    equal slices (a bit mask instead of the modulus reaches only the rows
    whose bits lie inside B - 1)."""
    n_keys = 4 * B
    keys = [O.fnv1a64(struct.pack("<q", i)) for i in range(n_keys)]
    rows = np.array([O.hashed_rows(k, 1, B, 0x5EED)[0] for k in keys])
    assert rows.min() >= 0 and rows.max() < B
    hit = np.unique(rows).size / B
    assert hit > 0.97, hit                  # 1 - e^-4 = 0.982 expected
    assert rows.max() >= B - 20
    n_slices = 45 if B == 45000 else 17
    counts = np.bincount(rows * n_slices // B, minlength=n_slices)
    exp = n_keys / n_slices
    chi2 = ((counts - exp) ** 2 / exp).sum()
    assert chi2 < 3 * n_slices, chi2        # about n_slices - 1 expected


# ---------------------------------------------------------------- softplus
def test_softplus_closed_forms():
    x = np.array([0.0, math.log(math.e - 1.0), 25.0, 100.0, -30.0, 1000.0], dtype=np.float64)
    y = O.softplus(x)
    assert y.dtype == np.float32
    assert y[0] == np.float32(math.log(2.0))
    assert y[1] == np.float32(1.0)                    # the "w_f = 1" initialisation
    assert y[2] == np.float32(25.0) and y[3] == np.float32(100.0) and y[5] == np.float32(1000.0)
    assert abs(float(y[4]) - math.exp(-30.0)) <= 1e-7 * math.exp(-30.0)
    # softplus(x) - softplus(-x) = x
    t = np.linspace(-15, 15, 301)
    d = O.softplus(t, np.float64) - O.softplus(-t, np.float64)
    assert np.max(np.abs(d - t)) < 1e-12


# ------------------------------------------------------- conditioning pins
def _small_index(seed=0, M=4, dsub=3, r=5, B=32, K=256):
    rng = np.random.default_rng(seed)
    return dict(
        C_pq=rng.standard_normal((M, K, dsub)).astype(np.float32),
        W=(0.1 * rng.standard_normal((M, r, K, dsub))).astype(np.float32),
        bank=(0.1 * rng.standard_normal((B, M * r))).astype(np.float32),
        M=M, dsub=dsub, r=r, B=B)


def test_identity_reduction_zero_bank_and_unit_weights():
    ix = _small_index()
    q = np.random.default_rng(1).standard_normal(ix["M"] * ix["dsub"]).astype(np.float32)
    zero = np.zeros_like(ix["bank"])
    alpha, w_f = O.select_codebook(q, [(0, 1, 5)], zero, 2, 3, None)
    assert np.all(alpha == 0) and not np.any(np.signbit(alpha))
    assert np.all(w_f == 1.0)
    C = O.conditioned_codebook(ix["C_pq"], ix["W"], alpha, ix["M"], ix["r"])
    assert np.array_equal(C.view(np.uint32), ix["C_pq"].view(np.uint32))
    lut_zero = O.build_lut(q, alpha, w_f, ix["C_pq"], ix["W"], ix["M"], ix["r"])
    lut_none = O.build_lut(q, None, None, ix["C_pq"], None, ix["M"], ix["r"])
    assert np.array_equal(lut_zero.view(np.uint32), lut_none.view(np.uint32))


def test_alpha_sums_hashed_rows_and_scales_exactly():
    ix = _small_index()
    q = np.arange(12, dtype=np.float32)
    clauses = [(0, -3, 10), (2, 0, 1)]
    rows = O.hashed_rows(O.fingerprint(q, clauses), 3, ix["B"], 11)
    alpha, _ = O.select_codebook(q, clauses, ix["bank"], 3, 11, None)
    expect = ((ix["bank"][rows[0]] + ix["bank"][rows[1]]) + ix["bank"][rows[2]])
    assert np.array_equal(alpha, expect)
    alpha2, _ = O.select_codebook(q, clauses, 2 * ix["bank"], 3, 11, None)
    assert np.array_equal(alpha2, 2 * alpha)


def test_delta_matches_library_contraction():
    ix = _small_index(seed=3)
    alpha = np.random.default_rng(4).standard_normal(ix["M"] * ix["r"])
    C = O.conditioned_codebook(ix["C_pq"], ix["W"], alpha, ix["M"], ix["r"], np.float64)
    delta = np.einsum("mt,mtcj->mcj", alpha.reshape(ix["M"], ix["r"]), ix["W"].astype(np.float64))
    np.testing.assert_allclose(C, ix["C_pq"].astype(np.float64) + delta, rtol=1e-13, atol=1e-13)


def test_lut_identity_is_textbook_adc_table():
    ix = _small_index(seed=5, M=6, dsub=4)
    q = np.random.default_rng(6).standard_normal(24).astype(np.float32)
    lut64 = O.build_lut(q, None, None, ix["C_pq"], None, 6, ix["r"], np.float64)
    lut32 = O.build_lut(q, None, None, ix["C_pq"], None, 6, ix["r"])
    for m in range(6):
        ref = cdist(q[None, m * 4:(m + 1) * 4].astype(np.float64),
                    ix["C_pq"][m].astype(np.float64), "sqeuclidean")[0]
        np.testing.assert_allclose(lut64[m], ref, rtol=1e-12, atol=1e-12)
        # fp32: dsub + 2 rounded non-negative terms
        assert np.all(np.abs(lut32[m] - ref) <= (4 + 3) * U32 * ref + 1e-30)


def test_lut_power_of_two_weight_scaling_is_exact():
    ix = _small_index(seed=7)
    rng = np.random.default_rng(8)
    q = rng.standard_normal(12).astype(np.float32)
    alpha = rng.standard_normal(ix["M"] * ix["r"]).astype(np.float32)
    w = O.softplus(rng.standard_normal(12))
    base = O.build_lut(q, alpha, w, ix["C_pq"], ix["W"], ix["M"], ix["r"])
    for s in (2.0, 0.5, 1024.0):
        scaled = O.build_lut(q, alpha, (w * np.float32(s)).astype(np.float32),
                             ix["C_pq"], ix["W"], ix["M"], ix["r"])
        assert np.array_equal(scaled, base * np.float32(s))


# ------------------------------------------------ ranking vs paper formula
def _conditioned_case(seed, N=300, M=4, dsub=3, r=5):
    ix = _small_index(seed=seed, M=M, dsub=dsub, r=r)
    rng = np.random.default_rng(seed + 100)
    codes = rng.integers(0, 256, (N, M), dtype=np.uint8)
    q = rng.standard_normal(M * dsub).astype(np.float32)
    alpha = rng.standard_normal(M * r).astype(np.float32)
    w = O.softplus(0.5 * rng.standard_normal(M * dsub), np.float64)
    return ix, codes, q, alpha, w


def test_distance_equals_weighted_q_norm_minus_paper_score():
    ix, codes, q, alpha, w = _conditioned_case(9)
    M, dsub, r = ix["M"], ix["dsub"], ix["r"]
    lut = O.build_lut(q, alpha, w, ix["C_pq"], ix["W"], M, r, np.float64)
    ids = np.arange(codes.shape[0])
    dist = O.adc_distances(lut, codes, ids, np.float64)
    # the score display of Section 2, stage 2, written term by term
    Wd = ix["W"].astype(np.float64)
    Cp = ix["C_pq"].astype(np.float64)
    a = alpha.astype(np.float64).reshape(M, r)
    qq = q.astype(np.float64)
    wq2 = float(np.sum(w * qq * qq))
    for v in range(0, codes.shape[0], 7):
        score = 0.0
        for m in range(M):
            c = int(codes[v, m])
            C_ifvs = Cp[m, c] + sum(a[m, t] * Wd[m, t, c] for t in range(r))
            for d in range(dsub):
                i = m * dsub + d
                score += 2.0 * w[i] * qq[i] * C_ifvs[d] - w[i] * C_ifvs[d] ** 2
        assert abs(dist[v] - (wq2 - score)) <= 1e-10 * max(1.0, abs(dist[v]))


def test_adc_equals_weighted_distance_to_reconstruction():
    ix, codes, q, alpha, w = _conditioned_case(10)
    M, dsub, r = ix["M"], ix["dsub"], ix["r"]
    C = ix["C_pq"].astype(np.float64) + np.einsum(
        "mt,mtcj->mcj", alpha.astype(np.float64).reshape(M, r), ix["W"].astype(np.float64))
    xhat = np.concatenate([C[m][codes[:, m]] for m in range(M)], axis=1)     # [N][D]
    ref = ((q.astype(np.float64)[None, :] - xhat) ** 2 * w[None, :]).sum(1)
    lut64 = O.build_lut(q, alpha, w, ix["C_pq"], ix["W"], M, r, np.float64)
    d64 = O.adc_distances(lut64, codes, np.arange(codes.shape[0]), np.float64)
    np.testing.assert_allclose(d64, ref, rtol=1e-12)
    # the fp32 decision path stays within the forward-error bound of its
    # (M + dsub + 2r + 6) rounded operations on non-negative sums; the
    # conditioned codebook's rounding enters through (q - C)^2 relative to
    # the squared magnitudes, bounded here by the sum of w (q^2 + C^2) terms.
    lut32 = O.build_lut(q, alpha, w.astype(np.float32), ix["C_pq"], ix["W"], M, r)
    d32 = O.adc_distances(lut32, codes, np.arange(codes.shape[0]))
    scale = ((q.astype(np.float64)[None, :] ** 2 + xhat ** 2) * w[None, :]).sum(1)
    assert np.all(np.abs(d32 - ref) <= (M + dsub + 2 * r + 6) * 4 * U32 * scale)


def test_lossless_pq_top_k_is_exact_filtered_knn():
    """N <= 256 vectors, each its own codeword in every subspace: identity-mode
    ADC is the exact squared L2 distance, so the oracle's top-k must be the
    exact filtered kNN of the raw vectors (scipy cdist + argsort)."""
    rng = np.random.default_rng(12)
    N, M, dsub = 200, 8, 4
    x = rng.standard_normal((N, M * dsub)).astype(np.float32)
    C_pq = np.zeros((M, 256, dsub), dtype=np.float32)
    for m in range(M):
        C_pq[m, :N] = x[:, m * dsub:(m + 1) * dsub]
    codes = np.tile(np.arange(N, dtype=np.uint8)[:, None], (1, M))
    attrs = rng.integers(0, 50, (2, N), dtype=np.int32)
    index = dict(codes=codes, C_pq=C_pq, attrs=attrs)
    for t in range(20):
        q = rng.standard_normal(M * dsub).astype(np.float32)
        lo = int(rng.integers(0, 40))
        clauses = [(0, lo, lo + 20), (1, 0, 35)]
        res = O.filtered_search(index, q, clauses, 10, conditioned=False)
        keep = np.flatnonzero((attrs[0] >= lo) & (attrs[0] < lo + 20) & (attrs[1] < 35))
        dd = cdist(q[None].astype(np.float64), x[keep].astype(np.float64), "sqeuclidean")[0]
        exact = keep[np.argsort(dd, kind="stable")[:10]]
        n = min(10, keep.size)
        assert list(res["ids"][:n]) == list(exact[:n])
        assert np.all(res["ids"][n:] == -1)


def test_conditioned_top_k_is_weighted_knn_over_reconstruction():
    ix, codes, q, alpha, w = _conditioned_case(13, N=250)
    M, r = ix["M"], ix["r"]
    C = ix["C_pq"].astype(np.float64) + np.einsum(
        "mt,mtcj->mcj", alpha.astype(np.float64).reshape(M, r), ix["W"].astype(np.float64))
    xhat = np.concatenate([C[m][codes[:, m]] for m in range(M)], axis=1)
    ref = ((q.astype(np.float64)[None, :] - xhat) ** 2 * w[None, :]).sum(1)
    lut = O.build_lut(q, alpha, w.astype(np.float32), ix["C_pq"], ix["W"], M, r)
    ids = np.arange(0, codes.shape[0], 2)              # a filtered subset
    d = O.adc_distances(lut, codes, ids)
    top, _ = O.select_topk(d, ids, 15)
    assert list(top) == list(ids[np.argsort(ref[ids], kind="stable")[:15]])


# ------------------------------------------------------------------ filter
def test_filter_brute_force_and_special_cases():
    rng = np.random.default_rng(14)
    attrs = rng.integers(-50, 50, (3, 777), dtype=np.int32)
    clauses = [(0, -10, 20), (2, 0, 1 << 40)]
    m = O.predicate_mask(attrs, clauses)
    for i in range(777):
        expect = all(lo <= int(attrs[c][i]) < hi for c, lo, hi in clauses)
        assert bool(m[i]) == expect
    assert O.predicate_mask(attrs, []).all()                      # no clause: TRUE
    assert not O.predicate_mask(attrs, [(1, 5, 5)]).any()         # lo == hi: empty
    assert not O.predicate_mask(attrs, [(1, 9, 2)]).any()         # lo > hi: empty
    big = O.predicate_mask(attrs, [(1, -(1 << 62), 1 << 62)])     # bounds beyond int32
    assert big.all()


def test_bitmap_layout_written_out():
    mask = np.zeros(70, dtype=bool)
    mask[[0, 31, 32, 69]] = True
    words = O.selection_bitmap(mask)
    assert words.dtype == np.uint32 and list(words) == [0x80000001, 0x00000001, 0x00000020]
    assert list(O.passing_ids(mask)) == [0, 31, 32, 69]


# ------------------------------------------------------------------ select
def test_topk_ties_padding_and_invariants():
    d = np.array([3.0, 1.0, 2.0, 1.0, 1.0, 5.0], dtype=np.float32)
    ids = np.array([10, 7, 3, 2, 9, 4])
    top, dist = O.select_topk(d, ids, 4)
    assert list(top) == [2, 7, 9, 3]
    assert list(dist) == [1.0, 1.0, 1.0, 2.0]
    top, dist = O.select_topk(d[:2], ids[:2], 4)
    assert list(top) == [7, 10, -1, -1] and np.isinf(dist[2:]).all()
    top, dist = O.select_topk(np.zeros(0, np.float32), np.zeros(0, np.int64), 3)
    assert list(top) == [-1, -1, -1]


def test_duplicate_codes_rank_by_smaller_id_and_permutation_invariance():
    rng = np.random.default_rng(15)
    N, M = 120, 4
    codes = rng.integers(0, 256, (N, M), dtype=np.uint8)
    codes[77] = codes[5]
    codes[101] = codes[5]
    C_pq = rng.standard_normal((M, 256, 2)).astype(np.float32)
    q = C_pq[:, codes[5], :][np.arange(M), np.arange(M)].reshape(-1).copy()   # x_hat of row 5
    attrs = np.zeros((1, N), dtype=np.int32)
    index = dict(codes=codes, C_pq=C_pq, attrs=attrs)
    res = O.filtered_search(index, q, [], 5, conditioned=False)
    assert list(res["ids"][:3]) == [5, 77, 101] and res["dist"][0] == 0.0
    # permuting the rows (carrying ids) does not change the answer
    perm = rng.permutation(N)
    lut = O.build_lut(q, None, None, C_pq, None, M, 0)
    d = O.adc_distances(lut, codes[perm], np.arange(N))
    top, _ = O.select_topk(d, perm, 5)
    assert list(top) == list(res["ids"])


def test_fp16_lut_is_nearest_binary16_and_widened_in_adc():
    ix = _small_index(seed=16)
    q = np.random.default_rng(17).standard_normal(12).astype(np.float32)
    l32 = O.build_lut(q, None, None, ix["C_pq"], None, ix["M"], ix["r"])
    l16 = O.build_lut(q, None, None, ix["C_pq"], None, ix["M"], ix["r"], lut_dtype="f16")
    assert l16.dtype == np.float16
    up = np.nextafter(l16, np.float16(np.inf)).astype(np.float64)
    dn = np.nextafter(l16, np.float16(-np.inf)).astype(np.float64)
    err = np.abs(l16.astype(np.float64) - l32)
    assert np.all(err <= np.abs(up - l32)) and np.all(err <= np.abs(dn - l32))
    codes = np.random.default_rng(18).integers(0, 256, (50, ix["M"]), dtype=np.uint8)
    d = O.adc_distances(l16, codes, np.arange(50))
    assert d.dtype == np.float32
    ref = sum(l16[m][codes[:, m]].astype(np.float64) for m in range(ix["M"]))
    np.testing.assert_allclose(d, ref, rtol=ix["M"] * U32)


# ------------------------------------------------------- exact filtered kNN
def test_exact_distances_within_fp32_bound_of_library_fp64():
    """fp32 sequential squared L2 against scipy's fp64 cdist: the forward
    error of 2D + 1 roundings of non-negative terms and differences."""
    rng = np.random.default_rng(31)
    for D in (3, 96, 128, 960):
        x = (rng.standard_normal((300, D)) + 0.5).astype(np.float32)
        q = rng.standard_normal(D).astype(np.float32)
        ids = rng.permutation(300)[:120]
        d32 = O.exact_distances(x, q, ids)
        d64 = cdist(q[None].astype(np.float64), x[ids].astype(np.float64), "sqeuclidean")[0]
        assert d32.dtype == np.float32
        assert np.all(np.abs(d32 - d64) <= (2 * D + 2) * U32 * d64)
        # fp64 mode is the definition to rounding of fp64
        d_hi = O.exact_distances(x, q, ids, dtype=np.float64)
        assert np.allclose(d_hi, d64, rtol=1e-12, atol=0)


def test_exact_distance_written_out_for_one_vector():
    """Two dimensions by hand: (1.5 - 0.25)^2 + (-2 - 1)^2 = 1.5625 + 9."""
    x = np.array([[1.5, -2.0]], dtype=np.float32)
    q = np.array([0.25, 1.0], dtype=np.float32)
    assert O.exact_distances(x, q, [0])[0] == np.float32(10.5625)


def test_exact_filtered_search_is_brute_force_knn():
    rng = np.random.default_rng(32)
    N, D = 500, 24
    x = rng.standard_normal((N, D)).astype(np.float32)
    attrs = rng.integers(0, 30, (2, N), dtype=np.int32)
    for t in range(15):
        q = rng.standard_normal(D).astype(np.float32)
        lo = int(rng.integers(0, 25))
        clauses = [(0, lo, lo + 6), (1, 0, 20)] if t % 3 else [(1, lo, lo + 1)]
        res = O.exact_filtered_search(x, attrs, q, clauses, 12)
        keep = np.flatnonzero(np.all([(attrs[c] >= a) & (attrs[c] < b) for c, a, b in clauses], axis=0))
        dd = cdist(q[None].astype(np.float64), x[keep].astype(np.float64), "sqeuclidean")[0]
        exact = keep[np.argsort(dd, kind="stable")[:12]]
        n = min(12, keep.size)
        assert res["n_pass"] == keep.size
        assert list(res["ids"][:n]) == list(exact[:n])
        assert np.all(res["ids"][n:] == -1) and np.all(np.isinf(res["dist"][n:]))


def test_exact_search_agrees_with_lossless_pq_adc_ranking():
    """With every vector its own codeword, identity-mode ADC and the exact
    search rank the same rows (both are the squared L2 distance, summed in
    different orders)."""
    rng = np.random.default_rng(33)
    N, M, dsub = 220, 6, 4
    x = rng.standard_normal((N, M * dsub)).astype(np.float32)
    C_pq = np.zeros((M, 256, dsub), dtype=np.float32)
    for m in range(M):
        C_pq[m, :N] = x[:, m * dsub:(m + 1) * dsub]
    codes = np.tile(np.arange(N, dtype=np.uint8)[:, None], (1, M))
    attrs = rng.integers(0, 10, (1, N), dtype=np.int32)
    index = dict(codes=codes, C_pq=C_pq, attrs=attrs)
    for t in range(10):
        q = rng.standard_normal(M * dsub).astype(np.float32)
        clauses = [(0, t % 5, t % 5 + 4)]
        a = O.filtered_search(index, q, clauses, 8, conditioned=False)
        b = O.exact_filtered_search(x, attrs, q, clauses, 8)
        assert list(a["ids"]) == list(b["ids"])
        assert np.allclose(a["dist"], b["dist"], rtol=1e-5)


def test_exact_search_ties_go_to_the_smaller_id():
    x = np.zeros((6, 4), dtype=np.float32)
    x[[1, 4, 5]] = 1.0
    attrs = np.zeros((1, 6), dtype=np.int32)
    res = O.exact_filtered_search(x, attrs, np.ones(4, dtype=np.float32), [], 4)
    assert list(res["ids"]) == [1, 4, 5, 0]


# ------------------------------------------------------------------- SDC
def test_sdc_table_is_library_codeword_distances():
    """Symmetric with a zero diagonal, and within the fp32 bound of scipy's
    fp64 squared distances between codewords."""
    rng = np.random.default_rng(41)
    C = rng.standard_normal((3, 256, 5)).astype(np.float32)
    T = O.sdc_table(C)
    for m in range(3):
        assert np.array_equal(T[m], T[m].T) and np.all(np.diag(T[m]) == 0)
        ref = cdist(C[m].astype(np.float64), C[m].astype(np.float64), "sqeuclidean")
        assert np.all(np.abs(T[m] - ref) <= (2 * 5 + 2) * U32 * ref)


def test_encode_query_is_nearest_codeword():
    rng = np.random.default_rng(42)
    M, dsub = 4, 6
    C = rng.standard_normal((M, 256, dsub)).astype(np.float32)
    for t in range(20):
        q = rng.standard_normal(M * dsub).astype(np.float32)
        codes = O.encode_query(q, C)
        for m in range(M):
            d = cdist(q[None, m * dsub:(m + 1) * dsub].astype(np.float64), C[m].astype(np.float64), "sqeuclidean")[0]
            assert codes[m] == int(np.argmin(d))
    # equal distances: the lower index
    C2 = np.zeros((1, 256, 2), dtype=np.float32)
    C2[0, 7] = [1, 0]
    C2[0, 3] = [0, 1]
    C2[0, 1:] += 50
    C2[0, 7] = [1, 0]
    C2[0, 3] = [0, 1]
    assert O.encode_query(np.zeros(2, dtype=np.float32), C2)[0] == 0       # codeword 0 is (0, 0)
    C2[0, 0] = [9, 9]
    assert O.encode_query(np.zeros(2, dtype=np.float32), C2)[0] == 3       # 3 and 7 tie at 1: lower index


def test_sdc_at_a_reconstruction_is_identity_adc():
    """A query equal to the reconstruction of codes c*: its code is c* and its
    SDC table is the identity-mode ADC table, bit for bit."""
    rng = np.random.default_rng(43)
    M, dsub = 8, 4
    C = rng.standard_normal((M, 256, dsub)).astype(np.float32)
    cstar = rng.integers(0, 256, M)
    q = np.concatenate([C[m, cstar[m]] for m in range(M)])
    assert list(O.encode_query(q, C)) == list(cstar)
    adc = O.build_lut(q, None, None, C, None, M, 0)
    assert np.array_equal(O.sdc_lut(q, C).view(np.uint32), adc.view(np.uint32))


def test_sdc_distance_is_distance_between_reconstructions():
    rng = np.random.default_rng(44)
    N, M, dsub = 300, 6, 3
    C = rng.standard_normal((M, 256, dsub)).astype(np.float32)
    codes = rng.integers(0, 256, (N, M)).astype(np.uint8)
    attrs = rng.integers(0, 10, (1, N), dtype=np.int32)
    index = dict(codes=codes, C_pq=C, attrs=attrs)
    rec = lambda c: np.concatenate([C[m, c[m]] for m in range(M)]).astype(np.float64)
    for t in range(6):
        q = rng.standard_normal(M * dsub).astype(np.float32)
        res = O.sdc_filtered_search(index, q, [(0, 2, 8)], 5)
        qc = O.encode_query(q, C)
        keep = np.flatnonzero((attrs[0] >= 2) & (attrs[0] < 8))
        d64 = np.array([((rec(qc) - rec(codes[v])) ** 2).sum() for v in keep])
        order = keep[np.lexsort((keep, d64))][:5]
        assert list(res["ids"]) == list(order)
        got = res["dist"].astype(np.float64)
        ref = np.sort(d64)[:5]
        assert np.all(np.abs(got - ref) <= 1e-5 * ref + 1e-6)


# --------------------------------------------------- reconstruct-then-exact
def test_reconstruction_written_out_and_exact_over_it():
    """x_hat of one row by hand; exact search over reconstructions ranks like
    identity-mode ADC (both are squared L2 to x_hat, summed in different
    orders) and returns distance 0 for a query equal to a reconstruction."""
    rng = np.random.default_rng(51)
    M, dsub, N = 4, 3, 400
    C = rng.standard_normal((M, 256, dsub)).astype(np.float32)
    codes = rng.integers(0, 256, (N, M)).astype(np.uint8)
    xh = O.reconstruct(codes, C)
    v = 17
    assert np.array_equal(xh[v], np.concatenate([C[0, codes[v, 0]], C[1, codes[v, 1]],
                                                 C[2, codes[v, 2]], C[3, codes[v, 3]]]))
    attrs = rng.integers(0, 8, (1, N), dtype=np.int32)
    index = dict(codes=codes, C_pq=C, attrs=attrs)
    for t in range(8):
        q = rng.standard_normal(M * dsub).astype(np.float32)
        a = O.filtered_search(index, q, [(0, 1, 6)], 7, conditioned=False)
        b = O.exact_filtered_search(xh, attrs, q, [(0, 1, 6)], 7)
        assert list(a["ids"]) == list(b["ids"])
    res = O.exact_filtered_search(xh, attrs, xh[v], [], 1)
    assert res["ids"][0] == v and res["dist"][0] == 0.0
