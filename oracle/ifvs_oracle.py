"""Plain, slow CPU oracle of the iFVS filtered vector search hot path.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``; never by the product path.

Every function restates a definition of the paper (iFVS, Al-Mamun, Rayhan,
Aref; VLDB 2026 workshop) and cites the passage it follows:

* Section 2 (iFVS), opening paragraph: the query-predicate pair is fingerprinted
  by ``h`` independent hash functions into a memory bank of ``B`` rows whose
  hashed rows are summed into alpha (M x r); the predicate is encoded into
  w_z (D); W has shape M x r x K x d.
* Section 2, first display: Delta = alpha . W, w_f = softplus(w_z),
  C_iFVS = C_PQ + Delta.
* Section 2, stage 1 (Filter): the predicate is evaluated over each vector's
  relational attributes to form the candidate pool P.
* Section 2, stage 2 (Rank), score display: each candidate is reconstructed
  from C_iFVS and scored with weights w_f.
* Section 2, stage 3 (Select): the top-k candidates by score are returned.
* Section 2, training paragraph: alpha = 0 and w_f = 1 reduce C_iFVS to C_PQ.
* Section 1, SQL listing: WHERE conjunction ... ORDER BY distance ... LIMIT K.
* Section 3.1 (workloads): the ground truth is the exact filtered top-k over
  the predicate-passing vectors; Section 3.2, pre-filtering baseline (i):
  exact L2 distances over the full-precision vectors of the candidate set.
* Section 3.2, pre-filtering baseline (ii): vectors reconstructed from their
  PQ codes, then exact L2 distances (exact filtered kNN over the
  reconstructions).
* Section 3.2, pre-filtering baselines (iv) and (v): symmetric distance
  computation (SDC) -- the query is quantized too, and a candidate's
  distance sums codeword-to-codeword distances.

Readings taken where the paper is silent (all listed in the design notes):

* score vs distance: the score display equals sum_i w_i q_i^2 minus the
  weighted squared distance sum_i w_i (q_i - xhat_i)^2, so ranking by largest
  score is ranking by smallest weighted distance; the oracle returns that
  distance (a non-negative number) and ranks ascending.
* Delta = alpha . W is the per-subspace contraction over the r directions:
  Delta[m,c,j] = sum_t alpha[m,t] W[m,t,c,j] (the only reading that yields an
  M x K x d tensor that can be added to C_PQ).
* fingerprint: FNV-1a-64 of the query's fp32 bytes followed by the predicate's
  clauses; hash function i maps the key to row
  SplitMix64(key XOR SplitMix64(seed + i)) mod B.  FNV-1a (Fowler, Noll, Vo)
  and SplitMix64 (Steele, Lea, Flood 2014) are published methods.
* predicate: a conjunction of half-open integer ranges lo <= attr[col] < hi.
* ties in the ranking go to the smaller vector id; fewer than k candidates pad
  with (id -1, distance +inf).
* arithmetic: the paper fixes no precision.  The ranking decides integers
  (ids), so the decision is taken in the kernel's precision, fp32, each
  operation rounded to nearest even with no fused multiply-add, subspaces and
  sub-dimensions summed in index order.  Every function also runs in fp64
  (``dtype=np.float64``) so the fp32 results can be checked against the
  definition in higher precision.

Parity pins (what ties this code to something other than itself) live in
``tests/test_oracle_*.py``.  Parity with the paper's *trained* conditioning
(its memory bank, W and predicate encoder) is unpinned: the paper publishes
neither the parameters nor a worked example.
"""
from __future__ import annotations

import struct
from typing import Iterable, Sequence

import numpy as np

__all__ = [
    "KSUB",
    "fnv1a64",
    "splitmix64",
    "fingerprint_bytes",
    "fingerprint",
    "hashed_rows",
    "softplus",
    "select_codebook",
    "predicate_mask",
    "selection_bitmap",
    "passing_ids",
    "conditioned_codebook",
    "build_lut",
    "adc_distances",
    "select_topk",
    "filtered_search",
    "exact_distances",
    "exact_filtered_search",
    "reconstruct",
    "encode_query",
    "sdc_table",
    "sdc_lut",
    "sdc_filtered_search",
]

KSUB = 256                      # codewords per subspace: 8-bit PQ codes
_MASK64 = (1 << 64) - 1
_FNV_OFFSET = 0xCBF29CE484222325
_FNV_PRIME = 0x100000001B3
_GOLDEN = 0x9E3779B97F4A7C15


# --------------------------------------------------------------------------
# Fingerprint of <q, f> into the memory bank (Section 2, opening paragraph)
# --------------------------------------------------------------------------
def fnv1a64(data: bytes) -> int:
    """FNV-1a, 64-bit: for each byte, xor it into the state, then multiply by
    the FNV prime modulo 2^64; the state starts at the FNV offset basis."""
    h = _FNV_OFFSET
    for byte in data:
        h ^= byte
        h = (h * _FNV_PRIME) & _MASK64
    return h


def splitmix64(x: int) -> int:
    """One SplitMix64 output for generator state ``x``: advance the state by
    the golden-ratio increment, then apply the two xor-shift-multiply rounds
    and the final xor-shift.  splitmix64(s), splitmix64(s + gamma), ... is the
    generator's output sequence from seed s."""
    z = (x + _GOLDEN) & _MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def fingerprint_bytes(q: np.ndarray, clauses: Sequence[tuple[int, int, int]]) -> bytes:
    """The byte string that identifies <q, f>: q as little-endian fp32 bit
    patterns, then the clause count as int32, then every clause as
    (col int32, lo int64, hi int64), all little-endian, in the given order."""
    q32 = np.ascontiguousarray(q, dtype="<f4")
    out = [q32.tobytes(), struct.pack("<i", len(clauses))]
    for col, lo, hi in clauses:
        out.append(struct.pack("<iqq", int(col), int(lo), int(hi)))
    return b"".join(out)


def fingerprint(q: np.ndarray, clauses: Sequence[tuple[int, int, int]]) -> int:
    return fnv1a64(fingerprint_bytes(q, clauses))


def hashed_rows(key: int, h: int, n_rows: int, hash_seed: int) -> list[int]:
    """The h bank rows of a fingerprint: hash function i is
    row_i = SplitMix64(key XOR SplitMix64(seed + i)) mod B."""
    rows = []
    for i in range(h):
        salt = splitmix64((hash_seed + i) & _MASK64)
        rows.append(splitmix64(key ^ salt) % n_rows)
    return rows


def softplus(w_z: np.ndarray, dtype=np.float32) -> np.ndarray:
    """w_f = softplus(w_z) = log(1 + e^x) (Section 2, first display), evaluated
    in fp64 and rounded once to fp32.  For x > 20, log1p(e^x) = x + log1p(e^-x)
    and the correction (< 2.1e-9) is below half an fp32 ulp of x, so x itself
    is the correctly rounded fp32 result; that branch also avoids overflow."""
    x = np.asarray(w_z, dtype=np.float64)
    y = np.empty_like(x)
    big = x > 20.0
    y[big] = x[big]
    y[~big] = np.log1p(np.exp(x[~big]))
    return y.astype(dtype)


def select_codebook(q, clauses, bank, h, hash_seed, w_z, dtype=np.float32):
    """Per-query conditioning: alpha = sum of the h hashed bank rows (summed
    in hash-function order, starting from +0; a row hit twice is added twice)
    and w_f = softplus(w_z).  ``bank`` None means no memory bank: alpha = 0
    (the identity of the training paragraph).  ``w_z`` None means w_f = 1.

    Returns (alpha [M*r], w_f [D]) in ``dtype``.
    """
    D = int(np.asarray(q).shape[0])
    if bank is None:
        alpha = None
    else:
        bank = np.asarray(bank)
        rows = hashed_rows(fingerprint(q, clauses), h, bank.shape[0], hash_seed)
        alpha = np.zeros(bank.shape[1], dtype=dtype)
        for r_i in rows:
            alpha = alpha + bank[r_i].astype(dtype)
    if w_z is None:
        w_f = np.ones(D, dtype=dtype)
    else:
        w_f = softplus(w_z, dtype)
    return alpha, w_f


# --------------------------------------------------------------------------
# Filter (Section 2, stage 1; SQL listing of Section 1)
# --------------------------------------------------------------------------
def predicate_mask(attrs: np.ndarray, clauses: Iterable[tuple[int, int, int]]) -> np.ndarray:
    """sel[i] is true iff every clause (col, lo, hi) holds: lo <= attr[col][i] < hi.
    ``attrs`` is column-major [n_attr][N] int32.  No clauses: every vector passes."""
    attrs = np.asarray(attrs)
    n = attrs.shape[1]
    mask = np.ones(n, dtype=bool)
    for col, lo, hi in clauses:
        a = attrs[col].astype(np.int64)
        mask &= (a >= lo) & (a < hi)
    return mask


def selection_bitmap(mask: np.ndarray) -> np.ndarray:
    """Pack a boolean selection into uint32 words, least significant bit
    first: vector i is bit (i mod 32) of word (i div 32); tail bits are 0."""
    mask = np.asarray(mask, dtype=bool)
    n = mask.shape[0]
    words = np.zeros((n + 31) // 32, dtype=np.uint32)
    idx = np.flatnonzero(mask)
    np.bitwise_or.at(words, idx >> 5, np.left_shift(np.uint32(1), (idx & 31).astype(np.uint32)))
    return words


def passing_ids(mask: np.ndarray) -> np.ndarray:
    """The candidate pool P as ascending vector ids."""
    return np.flatnonzero(np.asarray(mask, dtype=bool)).astype(np.int64)


# --------------------------------------------------------------------------
# Conditioned codebook and distance table (Section 2, first display; Rank)
# --------------------------------------------------------------------------
def conditioned_codebook(C_pq, W, alpha, M, r, dtype=np.float32):
    """C_iFVS = C_PQ + Delta with Delta[m,c,j] = sum_{t<r} alpha[m,t] W[m,t,c,j],
    the sum taken in t order starting from +0.  alpha None: C_iFVS = C_PQ.

    C_pq: [M][K][dsub]; W: [M][r][K][dsub]; alpha: [M*r]."""
    C_pq = np.asarray(C_pq).astype(dtype)
    if alpha is None:
        return C_pq.copy()
    W = np.asarray(W).astype(dtype)
    alpha = np.asarray(alpha).astype(dtype).reshape(M, r)
    C = np.empty_like(C_pq)
    for m in range(M):
        delta = np.zeros(C_pq.shape[1:], dtype=dtype)
        for t in range(r):
            delta = delta + alpha[m, t] * W[m, t]
        C[m] = C_pq[m] + delta
    return C


def build_lut(q, alpha, w_f, C_pq, W, M, r, dtype=np.float32, lut_dtype="f32"):
    """Per-query asymmetric distance table over the conditioned codebook:

        LUT[m][c] = sum_{j<dsub} w_f[m,j] * (q[m,j] - C_iFVS[m,c,j])^2,

    summed in j order from +0, each product and sum rounded in ``dtype``.
    Summing LUT[m][code_v[m]] over m gives the weighted squared distance
    between q and v reconstructed from C_iFVS, which is sum_i w_i q_i^2 minus
    the paper's score(v).  lut_dtype "f16" rounds the fp32 table to binary16
    (nearest even; beyond the binary16 range it becomes +inf)."""
    q = np.asarray(q).astype(dtype)
    D = q.shape[0]
    dsub = D // M
    C = conditioned_codebook(C_pq, W, alpha, M, r, dtype)
    w = np.ones(D, dtype=dtype) if w_f is None else np.asarray(w_f).astype(dtype)
    K = C.shape[1]
    lut = np.empty((M, K), dtype=dtype)
    for m in range(M):
        acc = np.zeros(K, dtype=dtype)
        for j in range(dsub):
            e = q[m * dsub + j] - C[m, :, j]
            acc = acc + w[m * dsub + j] * (e * e)
        lut[m] = acc
    if lut_dtype == "f16":
        return lut.astype(np.float32).astype(np.float16)
    if lut_dtype != "f32":
        raise ValueError(f"unknown lut_dtype {lut_dtype!r}")
    return lut


def adc_distances(lut, codes, ids, dtype=np.float32):
    """ADC over the candidates: d(v) = sum_{m<M} LUT[m][codes[v][m]], summed in
    m order from +0 in ``dtype`` (an fp16 table is widened entry by entry)."""
    lut = np.asarray(lut)
    codes = np.asarray(codes)
    ids = np.asarray(ids, dtype=np.int64)
    d = np.zeros(ids.shape[0], dtype=dtype)
    for m in range(lut.shape[0]):
        d = d + lut[m][codes[ids, m]].astype(dtype)
    return d


def select_topk(d, ids, k):
    """The k best candidates: ascending (distance, id); fewer than k candidates
    are padded with id -1 and distance +inf.  Returns (ids int32 [k],
    dist float32 [k]) for fp32 input (fp64 input keeps fp64 distances)."""
    d = np.asarray(d)
    ids = np.asarray(ids, dtype=np.int64)
    order = np.lexsort((ids, d))[:k]
    out_ids = np.full(k, -1, dtype=np.int32)
    out_d = np.full(k, np.inf, dtype=d.dtype if d.dtype == np.float64 else np.float32)
    out_ids[: order.shape[0]] = ids[order]
    out_d[: order.shape[0]] = d[order]
    return out_ids, out_d


# --------------------------------------------------------------------------
# One filtered query, end to end (Section 2, Filter -> Rank -> Select)
# --------------------------------------------------------------------------
def filtered_search(index: dict, q, clauses, k, w_z=None, lut_dtype="f32",
                    dtype=np.float32, conditioned=True):
    """Answer one filtered query the way Section 2 describes it.

    ``index`` holds: codes [N][M] uint8, C_pq [M][K][dsub], attrs [A][N] int32,
    and, for the conditioned mode, bank [B][M*r], W [M][r][K][dsub], r, h,
    hash_seed.  ``conditioned`` False (or no bank in the index) is the
    identity mode alpha = 0.  Returns a dict with every stage's output."""
    codes = np.asarray(index["codes"])
    M = codes.shape[1]
    r = int(index.get("r", 0))
    bank = index.get("bank") if conditioned else None
    alpha, w_f = select_codebook(q, clauses, bank, int(index.get("h", 0)),
                                 int(index.get("hash_seed", 0)), w_z, dtype)
    lut = build_lut(q, alpha, w_f, index["C_pq"], index.get("W"), M, r, dtype, lut_dtype)
    mask = predicate_mask(index["attrs"], clauses)
    ids = passing_ids(mask)
    d = adc_distances(lut, codes, ids, dtype)
    top_ids, top_d = select_topk(d, ids, k)
    return {"alpha": alpha, "w_f": w_f, "lut": lut, "mask": mask, "ids": top_ids,
            "dist": top_d, "n_pass": int(ids.shape[0])}


# --------------------------------------------------------------------------
# Exact filtered kNN over the full-precision vectors (Section 3.1 ground
# truth; Section 3.2, pre-filtering baseline (i))
# --------------------------------------------------------------------------
def exact_distances(x, q, ids, dtype=np.float32):
    """Squared L2 distance from q to each candidate's full-precision vector:
    d(v) = sum_{j<D} (x[v][j] - q[j])^2, summed in j order from +0 in
    ``dtype``, the difference, its square and each addition rounded
    separately."""
    x = np.asarray(x)
    q = np.asarray(q).astype(dtype)
    ids = np.asarray(ids, dtype=np.int64)
    d = np.zeros(ids.shape[0], dtype=dtype)
    for j in range(x.shape[1]):
        e = x[ids, j].astype(dtype) - q[j]
        d = d + e * e
    return d


def exact_filtered_search(x, attrs, q, clauses, k, dtype=np.float32):
    """Exact filtered kNN: the predicate-passing rows ranked by
    exact_distances, ascending (distance, id), padded to k with (-1, +inf)."""
    ids = passing_ids(predicate_mask(attrs, clauses))
    d = exact_distances(x, q, ids, dtype)
    top_ids, top_d = select_topk(d, ids, k)
    return {"ids": top_ids, "dist": top_d, "n_pass": int(ids.shape[0])}


# --------------------------------------------------------------------------
# Reconstruction from PQ codes (Section 3.2, pre-filtering baseline (ii):
# reconstruct, then exact_filtered_search over the reconstructions)
# --------------------------------------------------------------------------
def reconstruct(codes, C_pq):
    """x_hat[v] = concatenation over m of codeword C_pq[m][codes[v][m]]."""
    codes = np.asarray(codes).astype(np.int64)
    C = np.asarray(C_pq)
    M = C.shape[0]
    return np.concatenate([C[m][codes[:, m]] for m in range(M)], axis=1)


# --------------------------------------------------------------------------
# Symmetric distance computation (Section 3.2, pre-filtering baselines (iv)
# and (v)): both the query and the data are quantized
# --------------------------------------------------------------------------
def encode_query(q, C_pq, dtype=np.float32):
    """The query's PQ code: per subspace m, the codeword nearest to its
    sub-vector by squared L2 (summed in j order from +0 in ``dtype``), the
    lowest index among equal distances."""
    q = np.asarray(q).astype(dtype)
    C = np.asarray(C_pq).astype(dtype)
    M, K, dsub = C.shape
    codes = np.empty(M, dtype=np.int64)
    for m in range(M):
        acc = np.zeros(K, dtype=dtype)
        for j in range(dsub):
            e = q[m * dsub + j] - C[m, :, j]
            acc = acc + e * e
        codes[m] = int(np.argmin(acc))          # first minimum
    return codes


def sdc_table(C_pq, dtype=np.float32):
    """Codeword-to-codeword squared distances of every subspace:
    T[m][a][b] = sum_{j<dsub} (C[m][a][j] - C[m][b][j])^2, j order from +0."""
    C = np.asarray(C_pq).astype(dtype)
    M, K, dsub = C.shape
    T = np.empty((M, K, K), dtype=dtype)
    for m in range(M):
        acc = np.zeros((K, K), dtype=dtype)
        for j in range(dsub):
            e = C[m, :, j][:, None] - C[m, :, j][None, :]
            acc = acc + e * e
        T[m] = acc
    return T


def sdc_lut(q, C_pq, dtype=np.float32, lut_dtype="f32", table=None):
    """The query's symmetric distance table: LUT[m][c] = T[m][enc(q)_m][c],
    so that summing LUT[m][code_v[m]] over m (adc_distances) gives the SDC
    distance of v.  lut_dtype "f16" rounds it to binary16 as build_lut does."""
    T = sdc_table(C_pq, dtype) if table is None else table
    codes = encode_query(q, C_pq, dtype)
    lut = T[np.arange(T.shape[0]), codes]
    if lut_dtype == "f16":
        return lut.astype(np.float32).astype(np.float16)
    return lut


def sdc_filtered_search(index: dict, q, clauses, k, lut_dtype="f32", dtype=np.float32, table=None):
    """Filter, then rank the pool by SDC distance (ascending, ties to the
    smaller id), padded to k with (-1, +inf)."""
    codes = np.asarray(index["codes"])
    lut = sdc_lut(q, index["C_pq"], dtype, lut_dtype, table)
    ids = passing_ids(predicate_mask(index["attrs"], clauses))
    d = adc_distances(lut, codes, ids, dtype)
    top_ids, top_d = select_topk(d, ids, k)
    return {"lut": lut, "ids": top_ids, "dist": top_d, "n_pass": int(ids.shape[0])}
