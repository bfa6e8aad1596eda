"""The oracle's process pool answers exactly as single oracle calls do."""
import numpy as np
import pytest

import oracle as O
from oracle.pool import OraclePool, cpu_model, host_cores


def _index(rng, N=20_000, M=16, D=64):
    return dict(codes=rng.integers(0, 256, (N, M), dtype=np.uint8),
                C_pq=rng.standard_normal((M, 256, D // M)).astype(np.float32),
                attrs=rng.integers(0, 1000, (2, N), dtype=np.int32),
                bank=(rng.standard_normal((45_000, M * 4)) * 0.05).astype(np.float32),
                W=(rng.standard_normal((M, 4, 256, D // M)) * 0.05).astype(np.float32),
                r=4, h=3, hash_seed=11)


def test_pool_matches_single_calls():
    rng = np.random.default_rng(5)
    ox = _index(rng)
    D = 64
    tasks = []
    for i in range(24):
        cl = [(0, 10 * i, 10 * i + 300), (1, 0, 700)] if i % 3 else []
        wz = rng.standard_normal(D).astype(np.float32) if i % 2 else None
        tasks.append(((i, "x"), rng.standard_normal(D).astype(np.float32), cl, 7 + i % 5, wz,
                      "f16" if i % 4 == 0 else "f32", i % 5 != 0))
    with OraclePool(ox, 3) as pool:
        got = pool.search(tasks)
    assert [g[0] for g in got] == [t[0] for t in tasks]
    for (key, q, cl, k, wz, lt, cond), (key2, ids, dist, sec, enc_err) in zip(tasks, got):
        assert enc_err is None
        ref = O.filtered_search(ox, q, cl, k, w_z=wz, lut_dtype=lt, conditioned=cond)
        assert np.array_equal(ids, ref["ids"]), key
        assert np.array_equal(dist.view(np.uint32), ref["dist"].view(np.uint32)), key
        assert sec >= 0


def test_pool_reports_a_dead_worker():
    rng = np.random.default_rng(6)
    ox = _index(rng, N=1000)
    with OraclePool(ox, 1) as pool:
        pool._procs[0].kill()
        pool._procs[0].wait()
        with pytest.raises((RuntimeError, BrokenPipeError, OSError)):
            pool.search([((0,), np.zeros(64, np.float32), [], 5, None, "f32", False)])


def test_host_description():
    assert host_cores() >= 1
    assert isinstance(cpu_model(), str) and cpu_model()


def test_pool_encodes_when_asked():
    from oracle.ifvs_encoder_oracle import encode_predicate
    from workload import random_encoder
    rng = np.random.default_rng(8)
    ox = _index(rng)
    enc = random_encoder(2, 64, [1000, 1000], seed=4, hidden=32, heads=2, layers=1, ffn=32)
    enc_np = {k: (v.numpy() if hasattr(v, "numpy") else v) for k, v in enc.items() if k != "layers"}
    enc_np["layers"] = [{k: v.numpy() for k, v in p.items()} for p in enc["layers"]]
    preds = [[(0, 5, 300)], [], [(1, 0, 10), (0, 7, 700)]]
    wz = [encode_predicate(p, enc_np).astype(np.float32) for p in preds]
    wz[2] = wz[2] * np.float32(1.001)                          # one w_z 0.1% off
    tasks = [(i, rng.standard_normal(64).astype(np.float32), p, 5, wz[i], "f32", True, True)
             for i, p in enumerate(preds)]
    with OraclePool(ox, 2, encoder=enc) as pool:
        got = pool.search(tasks)
    assert got[0][4] < 1e-6 and got[1][4] < 1e-6
    assert 5e-4 < got[2][4] < 2e-3
    ref = O.filtered_search(ox, tasks[2][1], preds[2], 5, w_z=wz[2])
    assert np.array_equal(got[2][1], ref["ids"])
