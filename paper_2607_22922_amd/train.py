"""Train the filter-aware conditioning (memory bank and W) on a synthetic
workload and measure what it does to recall (Section 2, training paragraph;
Section 3's train / test split of the query workload).

Usage:
    python -m paper_2607_22922_amd.train [--config c4] [--bin 0.01] ...

Every step runs in the library: positives are the exact filtered top-k of
the full-precision vectors (ifvs_exact_search), hard negatives the best
conditioned-ADC results that are not positives (ifvs_filtered_search with
the current parameters, re-mined every epoch), and ifvs_train_step updates
the bank and W.  Training starts from alpha = 0 (a zero bank) and w_f = 1,
as the paper does; W starts from the workload's random values (with W = 0
no gradient reaches the bank).  Prints one JSON line: the step throughput,
the loss per epoch and recall@k of the conditioned search on the training
queries and on held-out test queries before and after training (the
identity mode, plain PQ, is the "before" value).
"""
from __future__ import annotations

import argparse
import json
import time

import torch


def _recall(ids, gt):
    hits = 0
    total = 0
    for a, b in zip(ids.tolist(), gt.tolist()):
        want = {v for v in b if v >= 0}
        hits += len(want & {v for v in a if v >= 0})
        total += len(want)
    return hits / max(1, total)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--config", default="c4")
    ap.add_argument("--N", type=int, default=None, help="base vectors (default: the config's)")
    ap.add_argument("--bin", type=float, default=0.01, help="selectivity bin of the training queries")
    ap.add_argument("--train-queries", type=int, default=2048)
    ap.add_argument("--test-queries", type=int, default=512)
    ap.add_argument("--batch", type=int, default=256)
    ap.add_argument("--epochs", type=int, default=20)
    ap.add_argument("--n-neg", type=int, default=32, help="hard negatives per query")
    ap.add_argument("--tau", type=float, default=1.0)
    ap.add_argument("--lam", type=float, default=0.1, help="anchor regularizer weight")
    ap.add_argument("--lr", type=float, default=20.0)
    args = ap.parse_args(argv)

    from paper_2607_22922_amd import ifvs as B
    from workload import make_workload

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    n_q = args.train_queries + args.test_queries
    t0 = time.time()
    w = make_workload(args.config, device=dev, n_queries=n_q, N=args.N, keep_x=True)
    torch.cuda.synchronize()
    gen_s = time.time() - t0
    k, batch = w.k, args.batch
    if args.bin not in w.bins:
        raise SystemExit(f"--bin must be one of {w.bins}")
    preds = w.preds[args.bin]
    bank0 = torch.zeros_like(w.bank)                       # alpha = 0 at the start
    idx = B.Index(w.codes, w.C_pq, w.attrs, bank0, w.W, w.r, w.h, w.hash_seed, max_batch=batch,
                  max_k=k + args.n_neg, cluster_cols=(0,))
    idx.load_vectors(w.x)
    w.x = None
    # Positives: the exact filtered top-k of every query.
    gt = torch.empty(n_q, k, dtype=torch.int32, device=dev)
    for b0 in range(0, n_q, batch):
        sl = slice(b0, min(n_q, b0 + batch))
        ids, _ = idx.exact_search(w.queries[sl].contiguous(), preds[sl], k)
        gt[sl] = ids
    train = range(0, args.train_queries)
    test = range(args.train_queries, n_q)

    def search(rows, kk, conditioned=True):
        out = torch.empty(len(rows), kk, dtype=torch.int32, device=dev)
        lo = rows.start
        for b0 in range(rows.start, rows.stop, batch):
            sl = slice(b0, min(rows.stop, b0 + batch))
            q = w.queries[sl].contiguous()
            if conditioned:
                alpha, wf = idx.select_codebook(q, preds[sl], None)
                lut = idx.build_lut(q, alpha, wf)
            else:
                lut = idx.build_lut(q)
            ids, _ = idx.search(preds[sl], lut, kk)
            out[b0 - lo:b0 - lo + ids.shape[0]] = ids
        return out

    def recall(rows, conditioned=True):
        ids = search(rows, k, conditioned)
        return _recall(ids, gt[rows.start:rows.stop])

    before = {"train": recall(train), "test": recall(test)}
    identity = {"train": recall(train, False), "test": recall(test, False)}
    losses, step_ms = [], 0.0
    n_steps = 0
    t_train = time.time()
    for epoch in range(args.epochs):
        mined = search(train, k + args.n_neg)             # current parameters
        ep_loss, ep_n = 0.0, 0
        for b0 in range(train.start, train.stop, batch):
            sl = slice(b0, min(train.stop, b0 + batch))
            pos = gt[sl]
            neg = mined[sl.start - train.start:sl.stop - train.start]
            # hard negatives: mined results that are not positives, best first
            is_pos = (neg[:, :, None] == pos[:, None, :]).any(dim=2) | (neg < 0)
            order = torch.argsort(is_pos.to(torch.int8), dim=1, stable=True)
            negs = torch.gather(neg, 1, order)[:, :args.n_neg]
            negs = torch.where(torch.gather(is_pos, 1, order)[:, :args.n_neg], torch.full_like(negs, -1), negs)
            cand = torch.cat([pos, negs], dim=1).contiguous()
            q = w.queries[sl].contiguous()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            loss, _ = idx.train_step(q, preds[sl], None, cand, k, args.tau, args.lam, args.lr)
            e1.record()
            torch.cuda.synchronize()
            step_ms += e0.elapsed_time(e1)
            n_steps += 1
            ep_loss += float(loss.sum())
            ep_n += loss.shape[0]
        losses.append(round(ep_loss / ep_n, 6))
    train_s = time.time() - t_train
    after = {"train": recall(train), "test": recall(test)}
    out = {
        "what": "iFVS conditioning trained with ifvs_train_step",
        "config": args.config, "N": w.N, "bin": args.bin, "k": k,
        "train_queries": args.train_queries, "test_queries": args.test_queries,
        "epochs": args.epochs, "batch": batch, "n_neg": args.n_neg, "tau": args.tau, "lam": args.lam,
        "lr": args.lr, "bank_rows": int(w.bank.shape[0]), "r": w.r, "h": w.h,
        "train_step_queries_per_s": n_steps * batch / (step_ms / 1e3) if step_ms > 0 else None,
        "train_step_ms": step_ms / max(1, n_steps),
        "training_wall_s": round(train_s, 2), "generation_s": round(gen_s, 1),
        "loss_per_epoch": losses,
        f"recall@{k}_identity": identity,
        f"recall@{k}_conditioned_before": before,
        f"recall@{k}_conditioned_after": after,
    }
    print(json.dumps(out), flush=True)
    return out


if __name__ == "__main__":
    main()
