#!/usr/bin/env python3
"""Benchmark of the iFVS filtered-search hot path on one MI355X.

Default workload (c4): 10M base vectors of 96 dims, PQ with 48 subspaces of
2 dims (48 B of codes per vector), one date-like int32 attribute uniform over
[0, 3650), range predicates at 0.1% / 1% / 10% / 50% selectivity, batches of
256 queries, k = 10, every step of the path in the conditioned mode (memory
bank, direction tensor, predicate weights).  Synthetic, seeded, generated on
the GPU (the paper's SIFT10M-style workload is not available here).
`--config c1|c2|c3|c5` measures the other synthetic workloads the same way
(1M x 128 with a range and a category clause, 1M x 960 with k = 100,
100M x 128, and the 10K-vector toy); rows are clustered by the range
attribute, or by (category, range attribute) where queries carry both.

One step = one batch of queries from each selectivity bin, each batch one
ifvs_query_batch call: encoder -> condition -> distance tables -> bounded
search (the list scan with the coarse bound where the planner takes it: the
10% and 50% bins on c4; the interval scan elsewhere).  `--separate-calls`
runs the four stages as four calls instead.  `value` is queries
per second over the timed steps, inputs resident in HBM.  In the timed
region only the scan kernel (the roofline kernel) and each bin's run of
batches are bracketed by HIP events; the per-stage breakdown and the
batch-to-batch spread come from passes of their own in which every kernel,
or every batch, is bracketed.

Prints one JSON line.  Progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "filtered QPS at recall@10 per selectivity bin; ADC scan HBM GB/s vs peak"
COUNTERS_FILE = os.path.join(ROOT, "profiles", "adc_scan_c4_counters.txt")
SCAN_SOURCES = [os.path.join(ROOT, "paper_2607_22922_amd", "csrc", f)
                for f in ("k_scan.hip", "k_listscan.hip", "k_coarse.hip", "topk_device.h")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def scan_source_hash() -> str:
    h = hashlib.sha256()
    for p in SCAN_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_counters():
    """Fabric-side bytes of the scan per launch, overall and per selectivity
    bin, from the committed rocprofv3 counter summary, if it was taken on the
    current scan source: {"mean": bytes, "by_bin": {bin: bytes}}."""
    if not os.path.exists(COUNTERS_FILE):
        return None
    kv = {}
    for line in open(COUNTERS_FILE):
        if "=" in line and not line.startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("scan_source_sha256_16") != scan_source_hash():
        return None
    try:
        by_bin = {}
        for item in kv["scan_fabric_bytes_per_launch_by_bin"].split(","):
            b, v = item.split(":")
            by_bin[b.strip()] = float(v)
        return {"mean": float(kv["scan_fabric_bytes_per_launch"]), "by_bin": by_bin}
    except (KeyError, ValueError):
        return None


SCAN_KERNEL_C4 = "scan_kernel<48, 1, float> and list_scan_kernel<48, float>"


def is_timed_scan_c4(kernel_name):
    """A timed scan kernel of the 10M-vector workload (the interval scan or
    the list scan, not their read-counting builds)."""
    return (("scan_kernel<48, 1, float" in kernel_name or "list_scan_kernel<48, float" in kernel_name)
            and ", true" not in kernel_name)


def summarize_counters(fetch_dir, write_dir, bins, steps, out_path, commands):
    """Writes the counter summary bench.py reads (see read_counters) from two
    rocprofv3 --pmc runs of `bench.py --steps S --warmup 0 ... --copy-calibration`
    (FETCH_SIZE, then WRITE_SIZE): the first 2 * S * len(bins) dispatches of
    the timed scan kernel are the stage pass and the timed pass, bins in
    order, S launches each; the copy kernel (1 GiB read, 1 GiB written)
    calibrates KiB to bytes."""
    import csv
    import glob

    def per_dispatch(d, counter):
        rows = []
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(path) as f:
                for r in csv.DictReader(f):
                    if r.get("Counter_Name") == counter:
                        rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
        agg = {}
        for did, kname, v in rows:
            a = agg.setdefault(did, [kname, 0.0])
            a[1] += v
        return [(did, agg[did][0], agg[did][1]) for did in sorted(agg)]

    fetch = per_dispatch(fetch_dir, "FETCH_SIZE")
    write = per_dispatch(write_dir, "WRITE_SIZE")
    copy_f = [v for _, kn, v in fetch if "neg" in kn.lower()]
    copy_w = [v for _, kn, v in write if "neg" in kn.lower()]
    gib_kib = float(1 << 20)
    f_fac = gib_kib / float(np.median(copy_f))
    w_fac = gib_kib / float(np.median(copy_w))
    n_timed = 2 * steps * len(bins)
    sf = [v for _, kn, v in fetch if is_timed_scan_c4(kn)][:n_timed]
    sw = [v for _, kn, v in write if is_timed_scan_c4(kn)][:n_timed]
    if len(sf) < n_timed or len(sw) < n_timed:
        raise RuntimeError(f"expected {n_timed} scan dispatches, found {len(sf)} / {len(sw)}")
    by_bin = {}
    for i, s in enumerate(bins):
        sel = [j for j in range(n_timed) if (j % (steps * len(bins))) // steps == i]
        by_bin[str(s)] = float(np.mean([(sf[j] * f_fac + sw[j] * w_fac) * 1024 for j in sel]))
    mean = float(np.mean([(sf[j] * f_fac + sw[j] * w_fac) * 1024 for j in range(n_timed)]))
    with open(out_path, "w") as f:
        f.write("# Fabric-side traffic of the ADC scan kernel (%s) on the 10M-vector\n" % SCAN_KERNEL_C4)
        f.write("# workload (10M x 96-d, PQ 48x2, clustered rows, batches of 256, k = 10), MI355X.\n")
        f.write("# Two rocprofv3 counter passes over the benchmark's stage pass and its timed pass\n")
        f.write("# (%d launches per bin each, bins %s), plus a copy kernel of known size (torch.neg\n"
                % (steps, "/".join(str(b) for b in bins)))
        f.write("# over 1 GiB fp32) for calibration.  Counters are KiB per dispatch.  FETCH_SIZE counts\n")
        f.write("# bytes the L2s request from the fabric: Infinity Cache hits are included (no gfx950\n")
        f.write("# counter separates them from HBM reads), so this is an upper bound on HBM traffic.\n")
        for c in commands:
            f.write("# command: %s\n" % c)
        f.write("copy_fetch_kib_per_dispatch = %.1f\n" % float(np.median(copy_f)))
        f.write("copy_write_kib_per_dispatch = %.1f\n" % float(np.median(copy_w)))
        f.write("fetch_factor = %.5f\nwrite_factor = %.5f\n" % (f_fac, w_fac))
        f.write("scan_fetch_kib_per_dispatch = %s\n" % ", ".join("%.0f" % v for v in sf))
        f.write("scan_write_kib_per_dispatch = %s\n" % ", ".join("%.0f" % v for v in sw))
        f.write("scan_fabric_bytes_per_launch_by_bin = %s\n"
                % ", ".join("%s:%.0f" % (b, v) for b, v in by_bin.items()))
        f.write("scan_fabric_bytes_per_launch = %.0f\n" % mean)
        f.write("scan_source_sha256_16 = %s\n" % scan_source_hash())


def clause_tensors(preds, device):
    """Clause lists as padded [nq][C] tensors (col, lo, hi); padding admits
    every value."""
    C = max(1, max(len(p) for p in preds))
    col = torch.zeros(len(preds), C, dtype=torch.int64)
    lo = torch.full((len(preds), C), -(1 << 62), dtype=torch.int64)
    hi = torch.full((len(preds), C), 1 << 62, dtype=torch.int64)
    for i, p in enumerate(preds):
        for j, (c, a, b) in enumerate(p):
            col[i, j], lo[i, j], hi[i, j] = c, a, b
    return col.to(device), lo.to(device), hi.to(device)


def exact_filtered_knn(name, N, attrs, queries, preds_by_bin, k):
    """Ground truth for recall: exact filtered kNN on the raw fp32 vectors
    (squared L2 in fp64), streamed over the regenerated base vectors so that
    no config needs its raw vectors kept.  Returns {bin: ids [nq][k]}."""
    from workload import base_chunks
    dev = queries.device
    nq = queries.shape[0]
    qd = queries.double()
    qn = (qd ** 2).sum(1)
    cl = {s: clause_tensors(p, dev) for s, p in preds_by_bin.items()}
    best = {s: (torch.full((nq, k), float("inf"), device=dev, dtype=torch.float64),
                torch.full((nq, k), -1, device=dev, dtype=torch.int64)) for s in preds_by_bin}
    for s0, xb in base_chunks(name, dev, N):
        rows = xb.shape[0]
        xd = xb.double()
        d = (xd ** 2).sum(1)[None, :] - 2.0 * (qd @ xd.t()) + qn[:, None]
        vals = attrs[:, s0:s0 + rows].long()
        for s, (col, lo, hi) in cl.items():
            ok = torch.ones(nq, rows, dtype=torch.bool, device=dev)
            for j in range(col.shape[1]):
                v = vals[col[:, j]]                                   # [nq][rows]
                ok &= (v >= lo[:, j, None]) & (v < hi[:, j, None])
            dd = torch.where(ok, d, torch.full_like(d, float("inf")))
            v_, i_ = torch.topk(dd, min(k, rows), dim=1, largest=False)
            bd, bi = best[s]
            cd = torch.cat([bd, v_], 1)
            ci = torch.cat([bi, i_ + s0], 1)
            v2, j2 = torch.topk(cd, k, dim=1, largest=False)
            best[s] = (v2, torch.gather(ci, 1, j2))
    return {s: torch.where(torch.isinf(v), torch.full_like(i, -1), i) for s, (v, i) in best.items()}


# Clustering of each workload's rows: the range attribute, or (category,
# range attribute) where the queries carry an equality on the category.
CLUSTER_COLS = {"c1": (0,), "c2": (1, 0), "c3": (0,), "c4": (0,), "c5": (1, 0)}

SCAN_WAVES = 8   # wavefronts per scan workgroup, each writing k partial keys per chunk

# The benchmark run the scan's counter passes profile: the timed pass and the
# stage pass only (3 launches per bin each), plus the calibration copy.
COARSE_ITERS = 20
COUNTER_RUN = ("--steps 3 --warmup 0 --plain-steps 0 --cpu-sample 0 --cpu-pool-queries 0 --recall-queries 0 "
               "--sdc-steps 0 --exact-steps 0 --host-steps 0 --no-lds-roof --copy-calibration")


def scan_bytes_interval(w, sorted_attr, preds, plan, k, lut_entry):
    """Algorithmic bytes of one interval-scan launch (one query per tile):
    the code tiles overlapping each query's row interval, its table, and its
    partial top-k lists (one per wavefront for every chunk written: with an
    absolute chunk grid only the cells the interval touches)."""
    lo = torch.tensor([p[0][1] for p in preds], device=sorted_attr.device, dtype=sorted_attr.dtype)
    hi = torch.tensor([p[0][2] for p in preds], device=sorted_attr.device, dtype=sorted_attr.dtype)
    r0 = torch.searchsorted(sorted_attr, lo)
    r1 = torch.searchsorted(sorted_attr, hi)
    nonempty = r1 > r0
    tiles = torch.where(nonempty, (r1 + 63) // 64 - r0 // 64, torch.zeros_like(r0))
    mw = (w.M + 3) // 4
    code = float(tiles.sum()) * 64 * mw * 4
    g = plan.get("grid_tiles", 0)
    if g and plan["splits"] * g >= (w.N + 63) // 64:   # absolute cells: one chunk per cell of the index
        cells = torch.where(nonempty, ((r1 + 63) // 64 - 1) // g - (r0 // 64) // g + 1, torch.zeros_like(r0))
        chunks = float(cells.sum())
    else:
        chunks = float(len(preds) * plan["splits"])
    return (code + len(preds) * w.M * 256 * lut_entry + chunks * SCAN_WAVES * k * 8,
            float((r1 - r0).sum()) * w.M)


def scan_union_bytes(w, sorted_attr, preds, plan, k, lut_entry, idx=None):
    """Bytes one scan launch must move between HBM and the chip at the
    least: every code tile that some query of the batch selects, read once
    (one-column intervals; otherwise every row some query selects, at M
    bytes), each query's table, and the partial top-k lists written."""
    mw = (w.M + 3) // 4
    if sorted_attr is not None:
        lo = torch.tensor([p[0][1] for p in preds], device=sorted_attr.device, dtype=sorted_attr.dtype)
        hi = torch.tensor([p[0][2] for p in preds], device=sorted_attr.device, dtype=sorted_attr.dtype)
        r0 = torch.searchsorted(sorted_attr, lo).cpu().numpy()
        r1 = torch.searchsorted(sorted_attr, hi).cpu().numpy()
        keep = r1 > r0
        t0, t1 = r0[keep] // 64, (r1[keep] + 63) // 64
        order = np.argsort(t0, kind="stable")
        tiles, end = 0, -1
        for a, b in zip(t0[order], t1[order]):
            a = max(a, end)
            if b > a:
                tiles += b - a
                end = b
        code = float(tiles) * 64 * mw * 4
        g = plan.get("grid_tiles", 0)
        if g and plan["splits"] * g >= (w.N + 63) // 64:
            chunks = float(np.sum(((r1[keep] + 63) // 64 - 1) // g - (r0[keep] // 64) // g + 1))
        else:
            chunks = float(len(preds) * plan["splits"])
    else:
        bm, _ = idx.filter(preds)
        any_row = bm.view(torch.int32)
        acc = torch.zeros_like(any_row[0])
        for i in range(any_row.shape[0]):
            acc |= any_row[i]
        rows = sum(bin(int(v) & 0xFFFFFFFF).count("1") for v in acc.cpu().tolist())
        code = float(rows) * w.M
        chunks = float(len(preds) * plan["splits"])
    return code + len(preds) * w.M * 256 * lut_entry + chunks * SCAN_WAVES * k * 8


def lds_roof(hist, rate):
    """LDS time of a scan's table reads: hist[n] reads with n active lanes,
    rate[n] such reads per second chip-wide (the probe).  Returns (lookups,
    seconds)."""
    lookups = sum(n * hist[n] for n in range(1, 65))
    secs = sum(hist[n] / rate[n] for n in range(1, 65) if hist[n])
    return lookups, secs


def exact_screen_bytes(w, sorted_attr, preds):
    """Bytes one screening pass of the exact search reads: every row of each
    32-query tile's hull (queries ordered by interval start, as the library
    orders them) as bf16 matrix-core fragments plus its squared norm."""
    lo = torch.tensor([p[0][1] for p in preds], device=sorted_attr.device, dtype=sorted_attr.dtype)
    hi = torch.tensor([p[0][2] for p in preds], device=sorted_attr.device, dtype=sorted_attr.dtype)
    r0 = torch.searchsorted(sorted_attr, lo)
    r1 = torch.searchsorted(sorted_attr, hi)
    order = torch.argsort(lo, stable=True)
    r0, r1 = r0[order], r1[order]
    rows = 0
    for t in range(0, len(preds), 32):
        a, b = r0[t:t + 32], r1[t:t + 32]
        keep = b > a
        if bool(keep.any()):
            rows += int(b[keep].max() - a[keep].min())
    return rows * (((w.D + 15) // 16) * 32 + 4)


def scan_bytes_passing(idx, w, preds, lut_entry):
    """Bytes a scan of this batch must read at the least: the codes of every
    (query, passing row) pair and each query's table.  Used where clustered
    intervals are composite (category, range) and the tile count of an
    interval is not a one-column search."""
    _, cnt = idx.filter(preds)
    useful = float(cnt.sum()) * w.M
    return useful + len(preds) * w.M * 256 * lut_entry, useful


def scan_bytes_bitmap(idx, w, preds, qt, splits, k, lut_entry):
    """Algorithmic bytes of one bitmap-scan launch (qt queries per tile): the
    code tiles any query of a tile selects, every query's bitmap words, its
    table and its partial top-k lists."""
    bm, cnt = idx.filter(preds)
    w64 = bm.view(torch.int64)
    n_tiles = w64.shape[1]
    pad = (-len(preds)) % qt
    if pad:
        w64 = torch.cat([w64, torch.zeros(pad, n_tiles, dtype=w64.dtype, device=w64.device)])
    any_t = (w64.view(-1, qt, n_tiles) != 0).any(1)
    mw = (w.M + 3) // 4
    code = float(any_t.sum()) * 64 * mw * 4
    nq = len(preds)
    return code + nq * (n_tiles * 8 + w.M * 256 * lut_entry + splits * SCAN_WAVES * k * 8), float(cnt.sum()) * w.M


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", choices=sorted(CLUSTER_COLS), default="c4",
                    help="synthetic workload (c4, the 10M-vector one, is the headline)")
    ap.add_argument("--queries", type=int, default=None,
                    help="queries drawn per bin (default: the config's count, at most 10,000)")
    ap.add_argument("--cpu-sample", type=int, default=2,
                    help="oracle queries per bin timed in one process on one core (0 = skip)")
    ap.add_argument("--cpu-pool-queries", type=int, default=None,
                    help="oracle queries per bin timed with one single-threaded process per core "
                         "(0 = skip; default 256 on c4, 16 on c1-c3, 4 on c5)")
    ap.add_argument("--cpu-pool-workers", type=int, default=16,
                    help="at most this many oracle processes (the host cores of the job)")
    ap.add_argument("--recall-queries", type=int, default=None,
                    help="queries per bin checked against exact filtered kNN (default 256; 100 on c1 and c5)")
    ap.add_argument("--plain-steps", type=int, default=None,
                    help="steps timed on the unclustered (bitmap) layout for comparison "
                         "(0 = skip; default 5 on c4, else 0)")
    ap.add_argument("--exact-steps", type=int, default=None,
                    help="batches per bin timed for exact filtered kNN over the full-precision vectors "
                         "(ifvs_exact_search; 0 = skip; default 4, 0 on c5)")
    ap.add_argument("--sdc-steps", type=int, default=4,
                    help="batches per bin timed with symmetric distance tables (ifvs_build_sdc_lut + the "
                         "same scan; 0 = skip)")
    ap.add_argument("--host-steps", type=int, default=4,
                    help="batches per bin timed with queries and weights uploaded from pinned host memory "
                         "and results downloaded inside each batch (the PCIe-inclusive rate; 0 = skip)")
    ap.add_argument("--lut", choices=["f32", "f16"], default="f32")
    ap.add_argument("--separate-calls", action="store_true",
                    help="run each batch as four calls (encoder, condition, tables, search) instead of "
                         "ifvs_query_batch; same results, each call stages the predicates again")
    ap.add_argument("--coarse", type=int, default=None,
                    help="coarse centroids of the list scan (ifvs_build_coarse; 0 = plain interval scan only; "
                         "default 2048 when D <= 128)")
    ap.add_argument("--no-recall-all", dest="recall_all", action="store_false",
                    help="skip recall over every query of every bin against ifvs_exact_search (needs the "
                         "exact-search leg)")
    ap.add_argument("--no-lds-roof", dest="lds_roof", action="store_false",
                    help="skip the read-counting pass and the LDS probe")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain copy kernel of known size (for counter calibration)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write the scan's counter summary (profiles/adc_scan_c4_counters.txt) from the "
                         "output folders of the two rocprofv3 counter runs of COUNTER_RUN, then exit")
    args = ap.parse_args()

    if args.summarize_counters:
        from workload.synth import CONFIGS
        cmds = [f"cd /tmp && export TMPDIR=/tmp; cd <repo>; rocprofv3 --pmc {c} --output-format csv -d "
                f"{d} -o run -- python3 bench.py {COUNTER_RUN}"
                for c, d in zip(("FETCH_SIZE", "WRITE_SIZE"), args.summarize_counters)]
        cmds.append("python3 bench.py --steps %d --summarize-counters %s %s"
                    % (args.steps, *args.summarize_counters))
        summarize_counters(*args.summarize_counters, CONFIGS["c4"]["bins"], args.steps, COUNTERS_FILE, cmds)
        print(open(COUNTERS_FILE).read())
        return

    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)

    from paper_2607_22922_amd import ifvs as B
    from workload import make_workload
    from workload.synth import CONFIGS, DESCRIPTIONS

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    name = args.config
    cfg = CONFIGS[name]
    n_q = args.queries if args.queries is not None else min(cfg["n_queries"], 10_000)
    batch, k = min(cfg.get("batch", 256), n_q), cfg["k"]
    if args.plain_steps is None:
        args.plain_steps = 5 if name == "c4" else 0
    if args.cpu_pool_queries is None:
        args.cpu_pool_queries = {"c4": 256, "c5": 4}.get(name, 16)
    if args.recall_queries is None:
        args.recall_queries = 100 if name in ("c1", "c5") else 256
    if args.exact_steps is None:
        args.exact_steps = 0 if name == "c5" else 4
    cols = CLUSTER_COLS[name]
    tile_bytes = cols == (0,)      # one-column intervals: bytes counted per code tile
    lut_dt = B.LUT_F16 if args.lut == "f16" else B.LUT_F32
    lut_entry = 2 if lut_dt == B.LUT_F16 else 4
    t0 = time.time()
    log(f"[bench] generating {name} on {dev}")
    w = make_workload(name, device=dev, n_queries=n_q, keep_x=False)
    torch.cuda.synchronize()
    log(f"[bench] generated in {time.time() - t0:.1f}s; loading indexes")
    clus = B.Index.from_workload(w, max_batch=batch, max_k=k, cluster_cols=cols)
    plain = B.Index.from_workload(w, max_batch=batch, max_k=k) if args.plain_steps > 0 else None
    for ix_ in (clus, plain):
        if ix_ is not None:
            ix_.load_encoder(w.enc)
    if args.coarse is None:
        args.coarse = 2048 if w.D <= 128 else 0
    coarse_build_s = None
    if args.coarse > 0:
        torch.cuda.synchronize()
        t_c = time.time()
        clus.build_coarse(args.coarse, COARSE_ITERS)
        coarse_build_s = time.time() - t_c
        log(f"[bench] coarse quantizer ({args.coarse} centroids, {COARSE_ITERS} k-means iterations) and "
            f"list order built in {coarse_build_s:.1f}s")
    n_batches = n_q // batch
    bins = w.bins

    # Marshalled inputs per (bin, batch): packed predicates; device buffers.
    packed = {s: [B.pack_predicates(w.preds[s][b * batch:(b + 1) * batch]) for b in range(n_batches)]
              for s in bins}
    alpha = torch.empty(batch, w.M * w.r, device=dev)
    wz = torch.empty(batch, w.D, device=dev)
    wf = torch.empty(batch, w.D, device=dev)
    lut = torch.empty(batch, w.M, 256, device=dev,
                      dtype=torch.float16 if lut_dt == B.LUT_F16 else torch.float32)
    ids = {s: torch.empty(batch, k, device=dev, dtype=torch.int32) for s in bins}
    dist = {s: torch.empty(batch, k, device=dev, dtype=torch.float32) for s in bins}
    stream = torch.cuda.current_stream()

    def run_batch(idx, s, b):
        sl = slice(b * batch, (b + 1) * batch)
        q = w.queries[sl]
        if not args.separate_calls:
            # one call: encoder, condition, tables and the search (the list
            # scan with the coarse bound where the planner picks it)
            idx.query_batch_into(q, packed[s][b], None, wz, alpha, wf, lut_dt, lut, k, ids[s], dist[s])
            return
        idx.encode_predicates_into(batch, packed[s][b], wz)
        idx.select_codebook_into(q, packed[s][b], wz, alpha, wf)
        idx.build_lut_into(q, alpha, wf, lut_dt, lut)
        if idx is clus and args.coarse > 0:
            # the tables' operands go with them: the search takes the list
            # scan with the coarse bound where the planner picks it
            idx.search_bounded_into(batch, packed[s][b], lut, lut_dt, alpha, wf, k, ids[s], dist[s])
        else:
            idx.search_into(batch, packed[s][b], lut, lut_dt, k, ids[s], dist[s])

    def timed_run(idx, steps, profile=2, warmup=None, per_batch=False):
        """W warmup steps, then `steps` timed steps.  profile 2 brackets the
        scan kernels' launches with HIP events on this stream, 3 only the
        list scan's, 1 every kernel (for the stage breakdown, in a separate
        pass).  Within the timed region the bins run one after another (each
        bin's `steps` batches together) so the kernel profile can be read per
        bin; a pair of events brackets each bin, and each batch only when
        per_batch is set (every event record costs the stream a few
        microseconds, so the timed pass leaves them out and a separate pass
        measures the spread).  Returns (total ms, per-bin [(b, ms)] -- each
        batch the bin's mean unless per_batch --, per-bin profile, whole
        profile, plans)."""
        for i in range(args.warmup if warmup is None else warmup):
            for s in bins:
                run_batch(idx, s, i % n_batches)
        torch.cuda.synchronize()
        idx.set_option(B.OPT_PROFILE, profile)
        idx.read_profile()
        ev = {s: [] for s in bins}
        prof_bin, plans = {}, {}
        torch.cuda.synchronize()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(stream)
        bin_ev = {}
        for s in bins:
            eb0, eb1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            eb0.record(stream)
            for i in range(steps):
                b = (args.warmup + i) % n_batches
                if per_batch:
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    run_batch(idx, s, b)
                    e1.record(stream)
                    ev[s].append((b, e0, e1))
                else:
                    run_batch(idx, s, b)
                    ev[s].append((b, None, None))
            eb1.record(stream)
            bin_ev[s] = (eb0, eb1)
            plans[s] = dict(idx.last_plan(), list_scan=idx.last_coarse())
            prof_bin[s] = idx.read_profile()           # waits for this bin's kernels
        stop.record(stream)
        torch.cuda.synchronize()
        total = start.elapsed_time(stop)
        idx.set_option(B.OPT_PROFILE, 0)
        prof = {st: (sum(prof_bin[s][st][0] for s in bins), sum(prof_bin[s][st][1] for s in bins))
                for st in prof_bin[bins[0]]}
        out = {}
        for s in bins:
            if per_batch:
                out[s] = [(b, a.elapsed_time(c)) for b, a, c in ev[s]]
            else:
                mean = bin_ev[s][0].elapsed_time(bin_ev[s][1]) / max(1, steps)
                out[s] = [(b, mean) for b, _, _ in ev[s]]
        return total, out, prof_bin, prof, plans

    # Stage breakdown (every kernel bracketed by events) in a short pass of its
    # own, first: it also names the dominant scan kernel (the interval or the
    # list scan, whichever takes more of the scan time), whose launches alone
    # the timed pass brackets with events (every event record costs the
    # stream a few microseconds); the other bins' scan times come from this
    # pass.
    _, _, stage_bin, stage_prof, stage_plans = timed_run(clus, min(args.steps, 3), profile=1,
                                                         warmup=min(2, args.warmup))
    pre_time = {}
    for s in bins:
        kk = "list_scan_kernel" if stage_plans[s].get("list_scan") else "scan_kernel"
        pre_time[kk] = pre_time.get(kk, 0.0) + stage_bin[s]["scan"][0]
    dom = max(pre_time, key=pre_time.get)
    total_ms, per_bin, prof_bin, prof, plans = timed_run(clus, args.steps,
                                                         profile=3 if dom == "list_scan_kernel" else 2)
    # The scan's table reads by active lanes, counted by the read-counting
    # build of the scan over the same batches (untimed), and the LDS's rate
    # for reads of each lane count, measured on this GPU.
    read_hist = {}
    if args.lds_roof:
        clus.set_option(B.OPT_COUNT_READS, 1)
        clus.read_scan_reads()
        for s in bins:
            for b, _ in per_bin[s]:
                run_batch(clus, s, b)
            read_hist[s] = clus.read_scan_reads()
        clus.set_option(B.OPT_COUNT_READS, 0)
        lds_rate = [0.0] + [B.probe_lds_gather(n) for n in range(1, 65)]
        log(f"[bench] LDS random reads per second (chip): 64 lanes {lds_rate[64]:.3e}, "
            f"32 {lds_rate[32]:.3e}, 8 {lds_rate[8]:.3e}, 1 {lds_rate[1]:.3e}")
    # Batch-to-batch spread (each batch bracketed by events) in a pass of its own.
    _, spread_bin, _, _, _ = timed_run(clus, args.steps, profile=0, warmup=0, per_batch=True)
    stage_steps = min(args.steps, 3)
    n_queries = args.steps * len(bins) * batch
    qps = n_queries / (total_ms / 1e3)
    log(f"[bench] clustered: {args.steps} steps in {total_ms:.1f} ms -> {qps:.0f} queries/s")

    sorted_attr = torch.sort(w.attrs[0].long()).values if tile_bytes else None
    fabric = read_counters() if name == "c4" else None
    bins_out = {}
    kind, bin_bytes, bin_lds, scan_src = {}, {}, {}, {}
    scan_bytes_total = useful_total = union_total = 0.0
    for s in bins:
        cache = {}
        for b, _ in per_bin[s]:
            if b not in cache:
                bp = w.preds[s][b * batch:(b + 1) * batch]
                cache[b] = ((scan_bytes_interval(w, sorted_attr, bp, plans[s], k, lut_entry) if tile_bytes
                             else scan_bytes_passing(clus, w, bp, lut_entry))
                            + (scan_union_bytes(w, sorted_attr, bp, plans[s], k, lut_entry, clus),))
            scan_bytes_total += cache[b][0]
            useful_total += cache[b][1]
            union_total += cache[b][2]
        ms = [m for _, m in per_bin[s]]
        sel = float(np.mean([v[1] / (w.M * w.N * batch) for v in cache.values()]))
        # per launch: the timed pass's events where they bracket this bin's
        # scan (the dominant kernel), else the stage pass's
        t_ms, t_n = prof_bin[s]["scan"]
        if t_n > 0:
            b_avg, scan_src[s] = t_ms / t_n, "timed pass"
        else:
            sm, sn = stage_bin[s]["scan"]
            b_avg, scan_src[s] = sm / max(1, sn), "stage pass (every kernel bracketed by events)"
        b_n = len(per_bin[s])
        b_ms = b_avg * b_n
        b_sec = b_avg / 1e3
        b_bytes = sum(cache[b][0] for b, _ in per_bin[s]) / max(1, b_n)
        b_gbps = b_bytes / b_sec / 1e9
        b_union = sum(cache[b][2] for b, _ in per_bin[s]) / max(1, b_n)
        is_list = bool(plans[s].get("list_scan"))
        kind[s] = "list_scan_kernel" if is_list else "scan_kernel"
        if is_list and s in read_hist:
            # the list scan reads the first three groups' code words of each
            # tile it sums and the other words of the tiles with a row live
            # after them (both counted by its counting build; a tile two
            # queries sum is counted twice), and the tables, and writes
            # partial lists (at most its job cap per query)
            tiles = read_hist[s][0] / max(1, b_n)
            whole = read_hist[s][65] / max(1, b_n)
            mw = (w.M + 3) // 4
            group = 8 if (w.M % 8 == 0 and w.M > 16) else (4 if w.M % 4 == 0 else w.M)
            pre = min(mw, (3 * group + 3) // 4)     # the list scan's kListPreGroups = 3
            b_union = (tiles * pre * 256 + whole * (mw - pre) * 256 + batch * w.M * 256 * lut_entry
                       + batch * plans[s]["splits"] * 8 * k * 8)
            b_bytes = b_union
        bin_bytes[s] = (b_union, b_bytes, b_n, b_ms)
        roofs = {"hbm": {"achieved_GBps": round(b_union / b_sec / 1e9, 1), "peak_GBps": HBM_PEAK_GBPS,
                         "frac": round(b_union / b_sec / 1e9 / HBM_PEAK_GBPS, 4),
                         "bytes_per_launch": b_union}}
        if is_list and s in read_hist:
            roofs["hbm"]["tiles_per_launch"] = read_hist[s][0] / max(1, b_n)
        if fabric is not None and str(s) in fabric["by_bin"]:
            fb = fabric["by_bin"][str(s)]
            roofs["hbm"]["fabric_bytes_per_launch"] = fb
            roofs["hbm"]["fabric_frac"] = round(fb / b_sec / 1e9 / HBM_PEAK_GBPS, 4)
        if s in read_hist:
            lk, lsec = lds_roof(read_hist[s], lds_rate)
            lk, lsec = lk / max(1, b_n), lsec / max(1, b_n)
            bin_lds[s] = (lk * b_n, lsec * b_n)
            roofs["lds"] = {"lookups_per_launch": lk,
                            "achieved_GBps": round(4 * lk / b_sec / 1e9, 1),
                            "peak_GBps": round(4 * lk / lsec / 1e9, 1) if lsec > 0 else None,
                            "frac": round(lsec / b_sec, 4),
                            "reads_per_launch": sum(read_hist[s][1:65]) / max(1, b_n),
                            "lanes_per_read": round(lk / max(1.0, sum(read_hist[s][1:65]) / max(1, b_n)), 2)}
        bound = max(roofs, key=lambda r: roofs[r]["frac"])
        roofs["bound"] = bound
        roofs["frac"] = roofs[bound]["frac"]
        spread = [m for _, m in spread_bin[s]]
        bins_out[str(s)] = {"qps": batch * len(ms) / (sum(ms) / 1e3),
                            "ms_per_batch": float(np.mean(ms)),
                            "ms_per_batch_p10_p90": [round(float(np.percentile(spread, 10)), 4),
                                                     round(float(np.percentile(spread, 90)), 4)],
                            "ms_per_batch_p10_p90_pass": "a separate pass with each batch bracketed by events",
                            "realized_selectivity": round(sel, 5),
                            "scan_ms": round(b_ms / max(1, b_n), 4),
                            "scan_ms_source": scan_src[s],
                            "scan_kernel": kind[s],
                            "scan_effective_GBps": round(b_gbps, 1),
                            "roofline": roofs,
                            "stage_ms_per_launch": {st: round(v[0] / max(1, v[1]), 4)
                                                   for st, v in stage_bin[s].items()},
                            "plan": plans[s]}
    # The roofline of the dominant kernel (named by the stage pass), its
    # launches timed in the timed pass.
    k_time = {}
    for s in bins:
        k_time[kind[s]] = k_time.get(kind[s], 0.0) + bin_bytes[s][3]
    dom_bins = [s for s in bins if kind[s] == dom]
    scan_ms = sum(prof_bin[s]["scan"][0] for s in dom_bins)
    scan_launches = sum(prof_bin[s]["scan"][1] for s in dom_bins)
    scan_avg_ms = scan_ms / max(1, scan_launches)
    union_per_launch = sum(bin_bytes[s][0] * bin_bytes[s][2] for s in dom_bins) / max(1, scan_launches)
    bytes_per_launch = sum(bin_bytes[s][1] * bin_bytes[s][2] for s in dom_bins) / max(1, scan_launches)
    effective = bytes_per_launch / (scan_avg_ms / 1e3) / 1e9
    hbm_achieved = union_per_launch / (scan_avg_ms / 1e3) / 1e9
    lds_lookups_total = sum(bin_lds[s][0] for s in dom_bins if s in bin_lds)
    lds_secs_total = sum(bin_lds[s][1] for s in dom_bins if s in bin_lds)
    if read_hist and lds_secs_total > 0:
        lds_frac = lds_secs_total / (scan_ms / 1e3)
        lds_achieved = 4 * lds_lookups_total / (scan_ms / 1e3) / 1e9
        lds_peak = 4 * lds_lookups_total / lds_secs_total / 1e9
    else:
        lds_frac = lds_achieved = lds_peak = None
    if lds_frac is not None and lds_frac > hbm_achieved / HBM_PEAK_GBPS:
        roof_bound, achieved, peak = "lds", lds_achieved, lds_peak
    else:
        roof_bound, achieved, peak = "hbm", hbm_achieved, HBM_PEAK_GBPS
    bytes_word = ("code tiles each query sums, counted per query"
                  if dom == "list_scan_kernel" and all(s in read_hist for s in dom_bins)
                  else "the queries' interval tiles, from HBM at least" if dom == "list_scan_kernel"
                  else "from HBM at least")
    log(f"[bench] {dom} (bins {dom_bins}): {scan_launches} launches, avg {scan_avg_ms:.3f} ms, "
        f"{union_per_launch / 1e6:.1f} MB/launch ({bytes_word}) -> {hbm_achieved:.0f} GB/s; "
        f"bound {roof_bound}: {achieved:.0f} of {peak:.0f} GB/s")

    plain_out = None
    if plain is not None:
        p_total, p_bins, _, p_prof, p_plans = timed_run(plain, args.plain_steps, profile=1)
        p_bytes = 0.0
        for s in bins:
            cache = {}
            for b, _ in p_bins[s]:
                if b not in cache:
                    pl = p_plans[s]
                    cache[b] = scan_bytes_bitmap(plain, w, w.preds[s][b * batch:(b + 1) * batch],
                                                 pl["qtile"], pl["splits"], k, lut_entry)[0]
                p_bytes += cache[b]
        p_scan_ms, p_launch = p_prof["scan"]
        plain_out = {
            "qps": args.plain_steps * len(bins) * batch / (p_total / 1e3),
            "bins_qps": {str(s): batch * len(v) / (sum(m for _, m in v) / 1e3) for s, v in p_bins.items()},
            "scan_avg_ms": p_scan_ms / max(1, p_launch),
            "scan_GBps": (p_bytes / max(1, p_launch)) / (p_scan_ms / max(1, p_launch) / 1e3) / 1e9,
            "stage_ms_per_step": {st: round(v[0] / args.plain_steps, 4) for st, v in p_prof.items()},
            "plan": p_plans[bins[-1]],
        }
        log(f"[bench] plain layout: {plain_out['qps']:.0f} queries/s, scan {plain_out['scan_GBps']:.0f} GB/s")
        # both layouts must return the same answers
        for s in bins:
            a_, f_ = clus.select_codebook(w.queries[:batch], w.preds[s][:batch],
                                          clus.encode_predicates(w.preds[s][:batch]))
            lt = clus.build_lut(w.queries[:batch], a_, f_, lut_dt)
            i1, d1 = clus.search(w.preds[s][:batch], lt, k, lut_dt)
            i2, d2 = plain.search(w.preds[s][:batch], lt, k, lut_dt)
            assert torch.equal(i1, i2) and torch.equal(d1.view(torch.int32), d2.view(torch.int32)), s

    # Recall@k of the identity mode (alpha = 0, w_f = 1: plain PQ ADC) and of
    # the synthetic conditioned mode, against exact filtered kNN.
    nr = min(args.recall_queries, batch)
    gt_all = {}
    gt_all_ids = {}
    if nr > 0:
        t_gt = time.time()
        gt_all = exact_filtered_knn(name, w.N, w.attrs, w.queries[:nr], {s: w.preds[s][:nr] for s in bins}, k)
        log(f"[bench] exact filtered kNN of {nr} queries x {len(bins)} bins in {time.time() - t_gt:.1f}s")
    for s in (bins if nr > 0 else []):
        q = w.queries[:nr]
        preds = w.preds[s][:nr]
        t_np = gt_all[s].cpu().numpy()
        gt_all_ids[str(s)] = gt_all[s]
        for mode in ("identity", "conditioned", "sdc"):
            if mode == "sdc":
                lt = clus.build_sdc_lut(q, lut_dt)
            elif mode == "identity":
                lt = clus.build_lut(q, None, None, lut_dt)
            else:
                a_, f_ = clus.select_codebook(q, preds, clus.encode_predicates(preds))
                lt = clus.build_lut(q, a_, f_, lut_dt)
            got, _ = clus.search(preds, lt, k, lut_dt)
            g_np = got.cpu().numpy()
            hits = 0.0
            for i in range(nr):
                truth = set(int(v) for v in t_np[i] if v >= 0)
                if truth:
                    hits += len(truth & set(int(v) for v in g_np[i] if v >= 0)) / len(truth)
            bins_out[str(s)][f"recall@{k}_{mode}"] = round(hits / nr, 4)
    log(f"[bench] bins: {json.dumps(bins_out)}")

    # PCIe-inclusive rate: the same step with the batch's query vectors
    # copied from pinned host memory at its start and the ids and distances
    # copied back at its end, all on the stream (the predicate weights come
    # from the encoder on the device, the predicates are host arrays already).
    host_out = None
    if args.host_steps > 0:
        hq = torch.empty(batch, w.D, pin_memory=True)
        hid = torch.empty(batch, k, dtype=torch.int32, pin_memory=True)
        hdi = torch.empty(batch, k, pin_memory=True)
        q_dev = torch.empty(batch, w.D, device=dev)
        host_src = {s: [w.queries[b * batch:(b + 1) * batch].cpu()
                        for b in range(min(n_batches, args.host_steps))] for s in bins}

        def run_host(s, b):
            hq.copy_(host_src[s][b])
            q_dev.copy_(hq, non_blocking=True)
            clus.encode_predicates_into(batch, packed[s][b], wz)
            clus.select_codebook_into(q_dev, packed[s][b], wz, alpha, wf)
            clus.build_lut_into(q_dev, alpha, wf, lut_dt, lut)
            clus.search_into(batch, packed[s][b], lut, lut_dt, k, ids[s], dist[s])
            hid.copy_(ids[s], non_blocking=True)
            hdi.copy_(dist[s], non_blocking=True)
            torch.cuda.current_stream().synchronize()     # the caller reads the results

        host_bins, host_total = {}, 0.0
        for s in bins:
            run_host(s, 0)                                 # warmup
            ms = []
            for i in range(args.host_steps):
                b = i % len(host_src[s])
                t_ = time.perf_counter()
                run_host(s, b)
                ms.append((time.perf_counter() - t_) * 1e3)
            host_total += sum(ms)
            host_bins[str(s)] = {"qps": batch * len(ms) / (sum(ms) / 1e3), "ms_per_batch": float(np.median(ms))}
        host_out = {"qps": args.host_steps * len(bins) * batch / (host_total / 1e3), "steps": args.host_steps,
                    "bytes_to_device_per_batch": batch * w.D * 4, "bytes_to_host_per_batch": batch * k * 8,
                    "timing": "host wall clock per batch, from the host-side copy into the pinned buffers to "
                              "the results in pinned host memory", "bins": host_bins}
        log(f"[bench] with host transfers: {host_out['qps']:.0f} queries/s; {json.dumps(host_bins)}")

    # Symmetric distance computation (Section 3.2, pre-filtering baselines
    # (iv)/(v)): the query is quantized too; its codeword-distance table
    # feeds the same scan.
    sdc_out = None
    if args.sdc_steps > 0:
        sdc_bins, sdc_total = {}, 0.0
        for s in bins:
            clus.build_sdc_lut_into(w.queries[:batch], lut_dt, lut)
            clus.search_into(batch, packed[s][0], lut, lut_dt, k, ids[s], dist[s])      # warmup
            ev_ = []
            for i in range(args.sdc_steps):
                b = i % n_batches
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                clus.build_sdc_lut_into(w.queries[b * batch:(b + 1) * batch], lut_dt, lut)
                clus.search_into(batch, packed[s][b], lut, lut_dt, k, ids[s], dist[s])
                e1.record(stream)
                ev_.append((e0, e1))
            torch.cuda.synchronize()
            ms = [a_.elapsed_time(c_) for a_, c_ in ev_]
            sdc_total += sum(ms)
            sdc_bins[str(s)] = {"qps": batch * len(ms) / (sum(ms) / 1e3), "ms_per_batch": float(np.median(ms))}
            if f"recall@{k}_sdc" in bins_out[str(s)]:
                sdc_bins[str(s)][f"recall@{k}"] = bins_out[str(s)][f"recall@{k}_sdc"]
        sdc_out = {"qps": args.sdc_steps * len(bins) * batch / (sdc_total / 1e3), "steps": args.sdc_steps,
                   "bins": sdc_bins}
        log(f"[bench] SDC: {sdc_out['qps']:.0f} queries/s; {json.dumps(sdc_bins)}")

    # Exact filtered kNN over the full-precision vectors (Section 3.2's
    # pre-filtering baseline (i), the ground truth of Section 3.1): whole
    # batches timed with events on the stream, every stage included.
    exact_out = None
    if args.exact_steps > 0:
        from workload import base_chunks
        x = torch.empty(w.N, w.D, device=dev)
        for s0, xb in base_chunks(name, dev, w.N):
            x[s0:s0 + xb.shape[0]] = xb
        clus.load_vectors(x)
        del x
        torch.cuda.synchronize()
        ex_ids = torch.empty(batch, k, device=dev, dtype=torch.int32)
        ex_d = torch.empty(batch, k, device=dev)
        ex_bins, ex_total = {}, 0.0
        for s in bins:
            clus.exact_search_into(w.queries[:batch], packed[s][0], k, ex_ids, ex_d)   # warmup
            ms = []
            for i in range(args.exact_steps):
                b = i % n_batches
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                clus.exact_search_into(w.queries[b * batch:(b + 1) * batch], packed[s][b], k, ex_ids, ex_d)
                e1.record(stream)
                ms.append((e0, e1))
            torch.cuda.synchronize()
            ms = [a.elapsed_time(c) for a, c in ms]
            ex_total += sum(ms)
            ex_bins[str(s)] = {"qps": batch * len(ms) / (sum(ms) / 1e3), "ms_per_batch": float(np.median(ms))}
            if tile_bytes:
                ex_bins[str(s)]["screen_bytes_per_pass"] = int(np.mean(
                    [exact_screen_bytes(w, sorted_attr, w.preds[s][(i % n_batches) * batch:(i % n_batches + 1) * batch])
                     for i in range(args.exact_steps)]))
            if str(s) in gt_all_ids:
                nr_ = gt_all_ids[str(s)].shape[0]
                clus.exact_search_into(w.queries[:batch], packed[s][0], k, ex_ids, ex_d)
                same = (ex_ids[:nr_].long() == gt_all_ids[str(s)]).all(1).float().mean()
                ex_bins[str(s)]["same_ids_as_fp64_ground_truth"] = round(float(same), 4)
        # Recall over every query of every bin, against the exact filtered
        # kNN of the full-precision vectors (ifvs_exact_search: fp32 squared
        # L2, ties to the smaller id), for each distance mode.
        if args.recall_all:
            t_all = time.time()
            for s in bins:
                hits = {m_: 0.0 for m_ in ("identity", "conditioned", "sdc")}
                counted = 0
                for b0 in range(0, n_q, batch):
                    sl = slice(b0, min(n_q, b0 + batch))
                    q = w.queries[sl]
                    preds = w.preds[s][sl]
                    gt, _ = clus.exact_search(q, preds, k)
                    valid = gt >= 0
                    n_gt = valid.sum(1)
                    use = n_gt > 0
                    counted += int(use.sum())
                    for mode in hits:
                        if mode == "sdc":
                            lt = clus.build_sdc_lut(q, lut_dt)
                        elif mode == "identity":
                            lt = clus.build_lut(q, None, None, lut_dt)
                        else:
                            a_, f_ = clus.select_codebook(q, preds, clus.encode_predicates(preds))
                            lt = clus.build_lut(q, a_, f_, lut_dt)
                        got, _ = clus.search(preds, lt, k, lut_dt)
                        inter = ((got[:, :, None] == gt[:, None, :]) & valid[:, None, :]).any(1).sum(1)
                        hits[mode] += float((inter[use].double() / n_gt[use].double()).sum())
                for mode, hsum in hits.items():
                    bins_out[str(s)][f"recall@{k}_{mode}_all"] = round(hsum / max(1, counted), 4)
                bins_out[str(s)]["recall_all_queries"] = counted
            torch.cuda.synchronize()
            log(f"[bench] recall over all {n_q} queries per bin against exact filtered kNN in "
                f"{time.time() - t_all:.1f}s")
        exact_out = {"qps": args.exact_steps * len(bins) * batch / (ex_total / 1e3), "steps": args.exact_steps,
                     "bins": ex_bins,
                     "note": "exact fp32 squared L2 over the predicate-passing full-precision vectors; "
                             "bf16 matrix-core screening with an error bound, exact scoring of survivors"}
        log(f"[bench] exact search: {exact_out['qps']:.0f} queries/s; {json.dumps(ex_bins)}")

    # Oracle on the host cores: a bounded sample of the same workload, in two
    # modes -- one process on one core, and one single-threaded process per
    # core -- each on the first queries of every bin, every answer compared
    # with the GPU's (ids and distance bits).
    cpu = None
    if args.cpu_sample > 0 or args.cpu_pool_queries > 0:
        from oracle.pool import OraclePool, cpu_model, host_cores
        ox = dict(codes=w.codes.cpu().numpy(), C_pq=w.C_pq.cpu().numpy(),
                  attrs=w.attrs.cpu().numpy(), bank=w.bank.cpu().numpy(), W=w.W.cpu().numpy(),
                  r=w.r, h=w.h, hash_seed=w.hash_seed)
        n_gpu = max(args.cpu_sample, args.cpu_pool_queries)
        n_gpu = min(n_gpu, batch)
        gpu_res = {}
        for s in bins:
            q = w.queries[:n_gpu]
            preds = w.preds[s][:n_gpu]
            wz_g = clus.encode_predicates(preds)
            a_, f_ = clus.select_codebook(q, preds, wz_g)
            lt = clus.build_lut(q, a_, f_, lut_dt)
            g_ids, g_d = clus.search(preds, lt, k, lut_dt)
            gpu_res[s] = (g_ids.cpu().numpy(), g_d.cpu().numpy(), q.cpu().numpy(), wz_g.cpu().numpy())

        def oracle_mode(workers, per_bin):
            # each task: the oracle encodes the predicate (checked against the
            # GPU's w_z), then answers the query from the GPU's w_z, so ids and
            # distance bits can be compared exactly
            tasks = [((s, i), gpu_res[s][2][i], w.preds[s][i], k, gpu_res[s][3][i], args.lut, True, True)
                     for s in bins for i in range(per_bin)]
            with OraclePool(ox, workers, encoder=w.enc) as pool:
                pool.search(tasks[:workers])                 # workers up, index mapped
                t_ = time.perf_counter()
                res = pool.search(tasks)
                wall = time.perf_counter() - t_
            agree = all(np.array_equal(ids_o, gpu_res[key[0]][0][key[1]]) and
                        np.array_equal(d_o.view(np.uint32), gpu_res[key[0]][1][key[1]].view(np.uint32))
                        for key, ids_o, d_o, *_ in res)
            return {"value": len(tasks) / wall, "unit": "queries/s", "cores": workers,
                    "queries": len(tasks), "wall_s": round(wall, 2),
                    "cpu_s": round(sum(r[3] for r in res), 2),
                    "ids_and_dist_bits_match_gpu": bool(agree),
                    "encoder_max_rel_err": max(r[4] for r in res)}

        model, avail = cpu_model(), host_cores()
        single = oracle_mode(1, min(args.cpu_sample, n_gpu)) if args.cpu_sample > 0 else None
        if single:
            log(f"[bench] oracle, 1 core: {single['value']:.3f} queries/s, results match: "
                f"{single['ids_and_dist_bits_match_gpu']}")
        multi = None
        if args.cpu_pool_queries > 0:
            workers = max(1, min(avail, args.cpu_pool_workers))
            multi = oracle_mode(workers, min(args.cpu_pool_queries, n_gpu))
            log(f"[bench] oracle, {workers} processes: {multi['value']:.3f} queries/s, results match: "
                f"{multi['ids_and_dist_bits_match_gpu']}")
        head = multi or single
        per = (min(args.cpu_pool_queries, n_gpu) if multi else min(args.cpu_sample, n_gpu))
        cpu = {"value": head["value"], "unit": "queries/s", "cores": head["cores"], "kind": "oracle",
               "sample": f"first {per} queries of each of the {len(bins)} bins of the same workload "
                         f"({head['queries']} queries), conditioned mode, "
                         + ("one single-threaded numpy process per core" if multi else "one numpy process")
                         + f", {head['wall_s']} s wall",
               "cpu_model": model, "affinity_cores": avail,
               "ids_and_dist_bits_match_gpu": head["ids_and_dist_bits_match_gpu"],
               "encoder_max_rel_err_vs_gpu": head["encoder_max_rel_err"],
               "single_core": single, "all_cores": multi}

    if args.copy_calibration:
        n_el = 1 << 28                                       # 1 GiB in, 1 GiB out
        src = torch.ones(n_el, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()

    traffic = None
    if fabric is not None and all(str(s) in fabric["by_bin"] for s in dom_bins):
        traffic = sum(fabric["by_bin"][str(s)] * prof_bin[s]["scan"][1] for s in dom_bins) / max(1, scan_launches)
    out = {
        "metric": METRIC,
        "value": qps,
        "unit": "queries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": total_ms / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.lut,
        "data": "synthetic",
        "config": {"workload": f"{name}: {DESCRIPTIONS[name]}", "batch": batch, "k": k,
                   "coarse_centroids": args.coarse, "coarse_build_s": coarse_build_s,
                   "bins": bins, "mode": "conditioned (predicate encoder -> w_z, memory bank, W)",
                   "calls_per_batch": ("4 (encode_predicates, select_codebook, build_lut, filtered_search_bounded)"
                                       if args.separate_calls else "1 (ifvs_query_batch)"),
                   "layout": ("rows clustered by the range attribute" if cols == (0,)
                              else "rows clustered by (category, range attribute)"),
                   "queries_per_step": len(bins) * batch,
                   "recall_queries_per_bin": nr,
                   "recall_ground_truth": (f"recall@k_<mode>: the first {nr} queries of each bin against exact "
                                           "filtered kNN of the raw vectors in fp64 (streamed); "
                                           "recall@k_<mode>_all: every query of each bin against "
                                           "ifvs_exact_search (fp32 exact filtered kNN)")},
        "bins": bins_out,
        "stage_ms_per_step": {st: round(v[0] / stage_steps, 4) for st, v in stage_prof.items()},
        "roofline": {"bound": roof_bound, "achieved": achieved, "peak": peak, "unit": "GB/s",
                     "frac": achieved / peak, "traffic": traffic,
                     "kernel": dom, "bins": dom_bins, "avg_launch_ms": scan_avg_ms,
                     "scan_ms_by_kernel": {kk: round(v / args.steps, 4) for kk, v in k_time.items()},
                     "hbm": {"achieved": hbm_achieved, "peak": HBM_PEAK_GBPS, "frac": hbm_achieved / HBM_PEAK_GBPS,
                             "bytes_per_launch": union_per_launch,
                             "bytes_definition": ("the code words the list scan reads: the first three groups' "
                                                  "words of each tile it sums, the rest of the tiles with a row "
                                                  "live after them (its counting build counts both; a tile several "
                                                  "queries sum counts once per query, the repeats mostly served by "
                                                  "L2 and Infinity Cache), + tables + partial lists written"
                                                  if dom == "list_scan_kernel" else
                                                  "code tiles some query of the batch selects, read once, + tables "
                                                  "+ partial lists written (the least a launch moves to and from "
                                                  "HBM)"),
                             "fabric_bytes_per_launch": traffic,
                             "fabric_definition": "rocprofv3 FETCH_SIZE x 2 + WRITE_SIZE (copy-kernel calibrated): "
                                                  "bytes the L2s request from the fabric, Infinity Cache hits "
                                                  "included; no counter on gfx950 separates those from HBM reads"},
                     "lds": ({"achieved": lds_achieved, "peak": lds_peak, "frac": lds_frac,
                              "definition": "4 bytes per table entry the scan reads from LDS (reads counted by "
                                            "active lanes in an untimed pass over the same batches) / scan time; "
                                            "peak: the LDS's measured rate for random 4-byte reads with the same "
                                            "mix of active lanes (ifvs_probe_lds_gather)"}
                             if lds_frac is not None else None),
                     "effective_GBps": effective,
                     "effective_definition": ("as bytes_per_launch" if dom == "list_scan_kernel" else
                                              "code tiles overlapping each query's row interval + table + partial "
                                              "lists, counted once per query (rows several queries share are "
                                              "re-read, mostly from L2)" if tile_bytes else
                                              "codes of every (query, passing row) pair + table"),
                     "effective_bytes_per_launch": bytes_per_launch,
                     "useful_bytes_per_launch": useful_total / max(1, scan_launches)},
        "plain_layout": plain_out,
        "exact_search": exact_out,
        "sdc": sdc_out,
        "host_transfers": host_out,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
