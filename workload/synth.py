"""Seeded synthetic workloads for filtered PQ search.

This module only draws inputs: base vectors from a Gaussian mixture, a PQ
codebook trained by Lloyd's k-means with the vectors' 8-bit codes, relational
attribute columns, predicates tuned to selectivity bins, query vectors and the
synthetic conditioning parameters (memory bank, direction tensor W, predicate
weights w_z).  It holds none of the search method's arithmetic (no predicate
evaluation, no hashing, no distance tables, no ranking): the HIP path and the
CPU oracle both consume what it returns.

The paper evaluates on SIFT1M / SIFT10M with 10K queries per selectivity bin
and predicates over fixed SIFT dimensions (Section 3.1); those datasets are not
available here, so these mixtures stand in for them, at the five sizes listed
in ``CONFIGS``.  Everything is drawn with ``torch.Generator`` from fixed seeds,
so one (config, device type) pair always yields the same arrays.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch

KSUB = 256

# name -> parameters.  Seeds follow 1000*c + {1 base, 2 queries, 3 predicates,
# 4 k-means, 5 conditioning}, c = 1..5.
CONFIGS = {
    "c1": dict(idx=1, N=10_000, D=128, M=16, comps=32, attrs=[("uniform", 1000)],
               bins=[0.10], n_queries=100, k=10, fixed_width=100),
    "c2": dict(idx=2, N=1_000_000, D=128, M=16, comps=256,
               attrs=[("uniform", 1000), ("zipf", 100)],
               bins=[0.01, 0.10, 0.50], n_queries=10_000, k=10),
    "c3": dict(idx=3, N=1_000_000, D=960, M=120, comps=128, attrs=[("uniform", 10_000)],
               bins=[0.01, 0.10, 0.50], n_queries=1_000, k=100),
    "c4": dict(idx=4, N=10_000_000, D=96, M=48, comps=1024, attrs=[("uniform", 3650)],
               bins=[0.001, 0.01, 0.10, 0.50], n_queries=10_000, k=10, batch=256),
    "c5": dict(idx=5, N=100_000_000, D=128, M=16, comps=4096,
               attrs=[("uniform", 1000), ("zipf", 1000)],
               bins=[0.001, 0.01, 0.10], n_queries=10_000, k=10),
}

DESCRIPTIONS = {
    "c1": "10K x 128-d, PQ 16x8, 1 uniform attr, 100 queries, 10% range, k=10",
    "c2": "1M x 128-d, PQ 16x8, uniform + Zipf(1.1, 100) attrs, 1/10/50%, k=10",
    "c3": "1M x 960-d, PQ 120x8, 1 uniform attr, 1/10/50%, k=100",
    "c4": "10M x 96-d, PQ 48x2, 1 date-like attr [0,3650), 0.1/1/10/50%, batch 256, k=10",
    "c5": "100M x 128-d, PQ 16x8, uniform + Zipf(1.1, 1000) attrs, 0.1/1/10%, k=10",
}

MIX_SIGMA = 0.3                 # isotropic std of every mixture component
KMEANS_ITERS = 20
KMEANS_SAMPLE = 200_000
BANK_ROWS = 4096                # memory-bank rows B (smallest bank of the paper's Table 2)
R_DIRS = 8                      # adjustment directions r
H_FUNCS = 2                     # hash functions h
PARAM_STD = 0.05                # std of synthetic bank and W entries
WZ_CENTER = math.log(math.e - 1.0)   # softplus(WZ_CENTER) = 1
WZ_STD = 0.1
ZIPF_S = 1.1
# Predicate encoder sizes (hidden width, heads, layers, feed-forward width).
ENC_HIDDEN, ENC_HEADS, ENC_LAYERS, ENC_FFN = 64, 4, 2, 128


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=torch.device(device).type)
    g.manual_seed(seed)
    return g


@dataclass
class Workload:
    name: str
    N: int
    D: int
    M: int
    dsub: int
    k: int
    bins: list
    codes: torch.Tensor            # [N][M] uint8
    C_pq: torch.Tensor             # [M][256][dsub] fp32
    attrs: torch.Tensor            # [A][N] int32, column-major
    domains: list                  # attribute value domains
    queries: torch.Tensor          # [nq][D] fp32 (shared by every bin)
    preds: dict                    # bin -> list of clause lists [(col, lo, hi), ...]
    w_z: dict                      # bin -> [nq][D] fp32
    bank: torch.Tensor             # [B][M*r] fp32
    W: torch.Tensor                # [M][r][256][dsub] fp32
    r: int = R_DIRS
    h: int = H_FUNCS
    hash_seed: int = 0
    enc: dict | None = None        # predicate encoder weights (random_encoder)
    x: torch.Tensor | None = None  # raw base vectors (None when not kept)
    cat_probs: torch.Tensor | None = None
    extra: dict = field(default_factory=dict)


# ---------------------------------------------------------------- vectors
def mixture_means(n_comp: int, D: int, seed: int, device) -> torch.Tensor:
    g = _gen(seed, device)
    return torch.rand(n_comp, D, generator=g, device=device) * 2.0 - 1.0


def mixture_draw(n: int, means: torch.Tensor, g: torch.Generator) -> torch.Tensor:
    comp = torch.randint(0, means.shape[0], (n,), generator=g, device=means.device)
    noise = torch.randn(n, means.shape[1], generator=g, device=means.device)
    return means[comp] + MIX_SIGMA * noise


def kmeans_pq(sample: torch.Tensor, M: int, seed: int, iters: int = KMEANS_ITERS) -> torch.Tensor:
    """Lloyd's k-means per subspace on ``sample`` [n][D]: K distinct seeded
    samples as the initial centroids, ``iters`` assignment/update rounds, an
    empty cluster keeps its centroid.  Returns C_pq [M][256][dsub] fp32."""
    n, D = sample.shape
    dsub = D // M
    g = _gen(seed, sample.device)
    perm = torch.randperm(n, generator=g, device=sample.device)[:KSUB]
    xs = sample.reshape(n, M, dsub).permute(1, 0, 2).contiguous()          # [M][n][dsub]
    C = xs[:, perm, :].clone()                                              # [M][K][dsub]
    chunk = max(1, (1 << 26) // (M * KSUB))
    for _ in range(iters):
        sums = torch.zeros_like(C, dtype=torch.float64)
        counts = torch.zeros(M, KSUB, dtype=torch.float64, device=sample.device)
        cn = (C * C).sum(-1)                                                # [M][K]
        for s in range(0, n, chunk):
            xb = xs[:, s:s + chunk, :]
            dist = cn[:, None, :] - 2.0 * torch.bmm(xb, C.transpose(1, 2).contiguous())
            a = dist.argmin(-1)                                             # [M][b]
            sums.scatter_add_(1, a[..., None].expand(-1, -1, dsub), xb.double())
            counts.scatter_add_(1, a, torch.ones_like(a, dtype=torch.float64))
        nz = counts > 0
        newC = (sums / counts.clamp(min=1)[..., None]).float()
        C = torch.where(nz[..., None], newC, C)
    return C.contiguous()


def pq_encode(x: torch.Tensor, C: torch.Tensor) -> torch.Tensor:
    """Nearest-centroid code per subspace (uint8 [n][M])."""
    n, D = x.shape
    M, K, dsub = C.shape
    xs = x.reshape(n, M, dsub).permute(1, 0, 2)
    cn = (C * C).sum(-1)
    out = torch.empty(M, n, dtype=torch.uint8, device=x.device)
    chunk = max(1, (1 << 26) // (M * K))
    Ct = C.transpose(1, 2).contiguous()
    for s in range(0, n, chunk):
        xb = xs[:, s:s + chunk, :].contiguous()
        dist = cn[:, None, :] - 2.0 * torch.bmm(xb, Ct)
        out[:, s:s + chunk] = dist.argmin(-1).to(torch.uint8)
    return out.t().contiguous()


# ------------------------------------------------------------- attributes
def zipf_probs(n_cat: int, s: float = ZIPF_S) -> torch.Tensor:
    """P(c) proportional to (c+1)^-s over categories 0..n_cat-1 (fp64)."""
    w = torch.arange(1, n_cat + 1, dtype=torch.float64) ** (-s)
    return w / w.sum()


def draw_attribute(kind: str, domain: int, n: int, g: torch.Generator, device) -> torch.Tensor:
    if kind == "uniform":
        return torch.randint(0, domain, (n,), generator=g, device=device, dtype=torch.int32)
    if kind == "zipf":
        cdf = torch.cumsum(zipf_probs(domain), 0).to(device)
        u = torch.rand(n, generator=g, device=device, dtype=torch.float64)
        return torch.searchsorted(cdf, u, right=True).clamp_(max=domain - 1).to(torch.int32)
    raise ValueError(kind)


# ------------------------------------------------------------- predicates
def _round_half_up(x: float) -> int:
    return int(math.floor(x + 0.5))


def make_predicates(cfg: dict, s: float, nq: int, seed: int) -> list:
    """Clause lists tuned to selectivity ``s``.

    One attribute: a range [lo, lo + w) with w = round(s * domain) (or the
    config's fixed width), lo uniform in [0, domain - w].
    Two attributes (uniform range, Zipf category): pick a category c uniformly
    among those with P(c) >= s / 0.9, equality c, range width
    round(s / P(c) * domain); when no category is that frequent, the category
    clause becomes the rank prefix [0, c) with the smallest cumulative mass
    >= s and the range width is scaled by that mass instead."""
    g = torch.Generator()
    g.manual_seed(seed)
    attrs = cfg["attrs"]
    dom0 = attrs[0][1]
    preds = []
    if len(attrs) == 1:
        w = cfg.get("fixed_width") or max(1, _round_half_up(s * dom0))
        lo = torch.randint(0, dom0 - w + 1, (nq,), generator=g).tolist()
        return [[(0, int(l), int(l) + w)] for l in lo]
    probs = zipf_probs(attrs[1][1])
    eligible = torch.nonzero(probs >= s / 0.9).flatten()
    if eligible.numel() == 0:
        cum = torch.cumsum(probs, 0)
        c_hi = int(torch.nonzero(cum >= s).flatten()[0]) + 1
        mass = float(cum[c_hi - 1])
        w = min(dom0, max(1, _round_half_up(s / mass * dom0)))
        lo = torch.randint(0, dom0 - w + 1, (nq,), generator=g).tolist()
        return [[(0, int(l), int(l) + w), (1, 0, c_hi)] for l in lo]
    pick = torch.randint(0, eligible.numel(), (nq,), generator=g)
    u = torch.rand(nq, generator=g, dtype=torch.float64)
    for i in range(nq):
        c = int(eligible[pick[i]])
        w = min(dom0, max(1, _round_half_up(s / float(probs[c]) * dom0)))
        lo = int(math.floor(float(u[i]) * (dom0 - w + 1)))
        preds.append([(0, lo, lo + w), (1, c, c + 1)])
    return preds


def make_attributes(cfg: dict, N: int, device="cpu") -> torch.Tensor:
    """The config's attribute columns, column-major [A][N] int32."""
    g_attr = _gen(1000 * cfg["idx"] + 7, device)
    cols = [draw_attribute(kind, dom, N, g_attr, device) for kind, dom in cfg["attrs"]]
    return torch.stack(cols).contiguous()


# ----------------------------------------------------------------- build
def base_chunks(name: str, device="cpu", N: int | None = None, chunk_rows: int = 1 << 20):
    """The config's base vectors in generation order: yields (first row,
    [rows][D] fp32) chunk by chunk, the same stream make_workload encodes, so
    the raw vectors of a large config can be regenerated (for ground truth)
    without being kept."""
    cfg = CONFIGS[name]
    Nn = int(N if N is not None else cfg["N"])
    c = cfg["idx"]
    device = torch.device(device)
    means = mixture_means(cfg["comps"], cfg["D"], 1000 * c + 0, device)
    g_base = _gen(1000 * c + 1, device)
    pos = 0
    while pos < Nn:
        rows = min(chunk_rows, Nn - pos)
        yield pos, mixture_draw(rows, means, g_base)
        pos += rows


def make_workload(name: str, device="cpu", n_queries: int | None = None, N: int | None = None,
                  keep_x: bool = True, chunk_rows: int = 1 << 20) -> Workload:
    """Draw a whole workload.  ``N`` / ``n_queries`` shrink a config for quick
    tests (the recipe is otherwise unchanged).  Base vectors are drawn and
    encoded in chunks of ``chunk_rows``; ``keep_x`` False drops them."""
    cfg = dict(CONFIGS[name])
    if N is not None:
        cfg["N"] = int(N)
    nq = int(n_queries if n_queries is not None else cfg["n_queries"])
    c = cfg["idx"]
    Nn, D, M = cfg["N"], cfg["D"], cfg["M"]
    dsub = D // M
    device = torch.device(device)

    means = mixture_means(cfg["comps"], D, 1000 * c + 0, device)
    # PQ training sample: the first base vectors, topped up by a seeded draw
    # of its own from the same mixture
    n_sample = min(Nn, KMEANS_SAMPLE)
    chunks = base_chunks(name, device, Nn, chunk_rows)
    _, first = next(chunks)
    if n_sample <= first.shape[0]:
        sample = first[:n_sample]
    else:
        sample = torch.cat([first, mixture_draw(n_sample - first.shape[0], means,
                                                _gen(1000 * c + 6, device))])
    C_pq = kmeans_pq(sample, M, 1000 * c + 4)

    codes = torch.empty(Nn, M, dtype=torch.uint8, device=device)
    xs = [] if keep_x else None
    pos, chunk = 0, first
    while chunk is not None:
        rows = chunk.shape[0]
        codes[pos:pos + rows] = pq_encode(chunk, C_pq)
        if keep_x:
            xs.append(chunk)
        pos, chunk = next(chunks, (None, None))
    x = torch.cat(xs) if keep_x else None

    attrs = make_attributes(cfg, Nn, device)

    g_q = _gen(1000 * c + 2, device)
    queries = mixture_draw(nq, means, g_q).contiguous()

    preds, w_z = {}, {}
    g_c = _gen(1000 * c + 5, device)
    bank = (torch.randn(BANK_ROWS, M * R_DIRS, generator=g_c, device=device) * PARAM_STD).contiguous()
    W = (torch.randn(M, R_DIRS, KSUB, dsub, generator=g_c, device=device) * PARAM_STD).contiguous()
    for b_i, s in enumerate(cfg["bins"]):
        preds[s] = make_predicates(cfg, s, nq, 1000 * c + 3 + 10 * b_i)
        w_z[s] = (WZ_CENTER + WZ_STD * torch.randn(nq, D, generator=g_c, device=device)).contiguous()

    cat_probs = zipf_probs(cfg["attrs"][1][1]) if len(cfg["attrs"]) > 1 else None
    domains = [d for _, d in cfg["attrs"]]
    enc = random_encoder(len(domains), D, domains, 1000 * c + 7, device)
    return Workload(name=name, N=Nn, D=D, M=M, dsub=dsub, k=cfg["k"], bins=list(cfg["bins"]),
                    codes=codes, C_pq=C_pq, attrs=attrs, domains=domains,
                    queries=queries, preds=preds, w_z=w_z, bank=bank, W=W,
                    hash_seed=0x5EED0000 + c, x=x, cat_probs=cat_probs, enc=enc)


def random_encoder(n_attr: int, D: int, domains, seed: int, device="cpu", hidden: int = ENC_HIDDEN,
                   heads: int = ENC_HEADS, layers: int = ENC_LAYERS, ffn: int = ENC_FFN) -> dict:
    """Seeded synthetic weights of the predicate encoder (the trained ones are
    not published).  Matrices are drawn N(0, 1/fan_in), layer-norm gains
    1 + N(0, 0.1^2), biases N(0, 0.1^2), embeddings N(0, 1); the output map
    is scaled so that w_z = WZ_CENTER + N(0, WZ_STD^2)-sized variations, the
    spread of the synthetic w_z above.  Bound normalization: offset 0 and
    scale 1 / domain per column (a column's values map into [0, 1))."""
    g = _gen(seed, device)
    H, F = hidden, ffn

    def rn(*shape, std=1.0):
        return (torch.randn(*shape, generator=g, device=device) * std).contiguous()

    def layer():
        return dict(ln1_g=1.0 + rn(H, std=0.1), ln1_b=rn(H, std=0.1),
                    Wq=rn(H, H, std=H ** -0.5), Wk=rn(H, H, std=H ** -0.5), Wv=rn(H, H, std=H ** -0.5),
                    bq=rn(H, std=0.1), bk=rn(H, std=0.1), bv=rn(H, std=0.1),
                    Wo=rn(H, H, std=H ** -0.5), bo=rn(H, std=0.1),
                    ln2_g=1.0 + rn(H, std=0.1), ln2_b=rn(H, std=0.1),
                    W1=rn(H, F, std=H ** -0.5), b1=rn(F, std=0.1), W2=rn(F, H, std=F ** -0.5), b2=rn(H, std=0.1))

    enc = dict(heads=heads,
               col_offset=torch.zeros(n_attr, dtype=torch.float64),
               col_scale=torch.tensor([1.0 / float(d) for d in domains], dtype=torch.float64),
               col_embed=rn(n_attr, H), feat_w=rn(2, H), feat_b=rn(H, std=0.1), cls=rn(H))
    enc["layers"] = [layer() for _ in range(layers)]
    enc.update(lnf_g=1.0 + rn(H, std=0.1), lnf_b=rn(H, std=0.1), out_w=rn(H, D, std=WZ_STD * H ** -0.5),
               out_b=torch.full((D,), WZ_CENTER, device=device))
    return enc


def random_index(N: int, M: int, dsub: int, n_attr: int, domain: int, seed: int,
                 device="cpu", r: int = R_DIRS, bank_rows: int = 64) -> dict:
    """Small unstructured index (uniform codes, Gaussian codebook) for edge
    cases: ragged N, odd shapes, constructed ties."""
    g = _gen(seed, device)
    return dict(
        codes=torch.randint(0, KSUB, (N, M), generator=g, device=device, dtype=torch.uint8),
        C_pq=torch.randn(M, KSUB, dsub, generator=g, device=device),
        attrs=torch.randint(0, domain, (n_attr, N), generator=g, device=device, dtype=torch.int32),
        bank=torch.randn(bank_rows, M * r, generator=g, device=device) * PARAM_STD,
        W=torch.randn(M, r, KSUB, dsub, generator=g, device=device) * PARAM_STD,
        r=r, h=H_FUNCS, hash_seed=seed,
    )
