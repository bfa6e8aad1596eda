"""A process pool that runs the oracle's filtered search over many queries.

TEST INFRASTRUCTURE ONLY, like the rest of this package: used by the
full-size parity tests and by the benchmark's CPU baseline.  It adds no
arithmetic: every query is answered by ``filtered_search`` exactly as a
single call would answer it; the pool only spreads queries over host cores.

Each worker is a fresh ``python -m oracle.pool`` child process (it imports
numpy and the oracle, nothing of the parent's program), limited to one
BLAS/OpenMP thread, that reads pickled tasks on stdin and writes results on
stdout; the parent hands a worker its next task as soon as it returns one.
A worker that dies makes ``search`` raise.  The index arrays are written
once to a temporary directory as ``.npy`` files and memory-mapped read-only
by every worker, so a 1.6 GB code array is held once in the page cache, not
once per worker.

With an encoder (a dict of predicate-encoder weights), a task may also ask
the worker to encode its predicate with ``encode_predicate`` before the
search (the oracle then does every step of a conditioned query); the
search itself uses the w_z the task carries, and the worker reports how far
the oracle's own w_z is from it.
"""
from __future__ import annotations

import os
import pickle
import selectors
import shutil
import struct
import subprocess
import sys
import tempfile
import time

import numpy as np

_ARRAYS = ("codes", "C_pq", "attrs", "bank", "W")
_SCALARS = ("r", "h", "hash_seed")
_THREAD_VARS = ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS", "NUMEXPR_NUM_THREADS")
_ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def host_cores() -> int:
    """Cores this process may run on (its CPU affinity set)."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def cpu_model() -> str:
    """The host CPU's model name from /proc/cpuinfo ("unknown" if absent)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _send(f, obj) -> None:
    data = pickle.dumps(obj, protocol=pickle.HIGHEST_PROTOCOL)
    f.write(struct.pack("<Q", len(data)) + data)
    f.flush()


def _recv(f):
    head = f.read(8)
    if len(head) < 8:
        return None
    (n,) = struct.unpack("<Q", head)
    data = f.read(n)
    if len(data) < n:
        return None
    return pickle.loads(data)


class OraclePool:
    """``workers`` single-threaded processes answering filtered queries with
    the oracle over one index (a dict as ``filtered_search`` takes it).
    Use as a context manager; ``search`` returns results in task order."""

    def __init__(self, index: dict, workers: int | None = None, encoder: dict | None = None):
        self.workers = max(1, int(workers if workers is not None else host_cores()))
        self._dir = tempfile.mkdtemp(prefix="oracle_pool_")
        if encoder is not None:
            with open(os.path.join(self._dir, "encoder.pkl"), "wb") as f:
                pickle.dump(_to_numpy(encoder), f)
        for name in _ARRAYS:
            a = index.get(name)
            if a is not None:
                np.save(os.path.join(self._dir, name + ".npy"), np.ascontiguousarray(a))
        with open(os.path.join(self._dir, "scalars.pkl"), "wb") as f:
            pickle.dump({s: int(index.get(s, 0) or 0) for s in _SCALARS}, f)
        env = dict(os.environ)
        for v in _THREAD_VARS:
            env[v] = "1"
        env["PYTHONPATH"] = _ROOT + (os.pathsep + env["PYTHONPATH"] if env.get("PYTHONPATH") else "")
        self._procs = [subprocess.Popen([sys.executable, "-m", "oracle.pool", self._dir], env=env,
                                        stdin=subprocess.PIPE, stdout=subprocess.PIPE, cwd=_ROOT)
                       for _ in range(self.workers)]

    def search(self, tasks, progress=None):
        """tasks: iterable of (key, q [D], clauses, k, w_z [D] or None,
        lut_dtype, conditioned[, encode]).  Returns [(key, ids, dist, seconds,
        enc_err)] in task order, enc_err = max over dimensions of
        |w_z - oracle w_z| / (|oracle w_z| + 0.01) for tasks that encode, else
        None; ``progress(done, total)`` is called as results arrive."""
        tasks = list(tasks)
        out = [None] * len(tasks)
        nxt = 0
        sel = selectors.DefaultSelector()
        busy = 0
        for i, p in enumerate(self._procs):
            if nxt < len(tasks):
                _send(p.stdin, (nxt, tasks[nxt]))
                sel.register(p.stdout, selectors.EVENT_READ, i)
                nxt += 1
                busy += 1
        done = 0
        while busy:
            for key, _ in sel.select():
                p = self._procs[key.data]
                r = _recv(p.stdout)
                if r is None:
                    raise RuntimeError(f"oracle worker {p.pid} ended (exit status {p.poll()})")
                pos, res = r
                out[pos] = res
                done += 1
                if progress is not None:
                    progress(done, len(tasks))
                if nxt < len(tasks):
                    _send(p.stdin, (nxt, tasks[nxt]))
                    nxt += 1
                else:
                    sel.unregister(p.stdout)
                    busy -= 1
        sel.close()
        return out

    def close(self) -> None:
        for p in self._procs:
            try:
                p.stdin.close()
            except OSError:
                pass
        for p in self._procs:
            try:
                p.wait(timeout=30)
            except subprocess.TimeoutExpired:
                p.kill()
                p.wait()
        self._procs = []
        shutil.rmtree(self._dir, ignore_errors=True)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
        return False


def _to_numpy(obj):
    if isinstance(obj, dict):
        return {k: _to_numpy(v) for k, v in obj.items()}
    if isinstance(obj, (list, tuple)):
        return [_to_numpy(v) for v in obj]
    if hasattr(obj, "detach"):
        return obj.detach().cpu().numpy()
    return obj


def _worker(root: str) -> None:
    from oracle.ifvs_encoder_oracle import encode_predicate
    from oracle.ifvs_oracle import filtered_search
    with open(os.path.join(root, "scalars.pkl"), "rb") as f:
        index = pickle.load(f)
    enc = None
    if os.path.exists(os.path.join(root, "encoder.pkl")):
        with open(os.path.join(root, "encoder.pkl"), "rb") as f:
            enc = pickle.load(f)
    for name in _ARRAYS:
        path = os.path.join(root, name + ".npy")
        index[name] = np.load(path, mmap_mode="r") if os.path.exists(path) else None
    fin, fout = sys.stdin.buffer, sys.stdout.buffer
    while True:
        msg = _recv(fin)
        if msg is None:
            return
        pos, task = msg
        key, q, clauses, k, w_z, lut_dtype, conditioned = task[:7]
        encode = len(task) > 7 and bool(task[7])
        t0 = time.perf_counter()
        enc_err = None
        if encode:
            ref = encode_predicate(clauses, enc)
            enc_err = float(np.max(np.abs(np.asarray(w_z, dtype=np.float64) - ref) / (np.abs(ref) + 0.01)))
        res = filtered_search(index, q, clauses, k, w_z=w_z, lut_dtype=lut_dtype, conditioned=conditioned)
        _send(fout, (pos, (key, res["ids"], res["dist"], time.perf_counter() - t0, enc_err)))


if __name__ == "__main__":
    _worker(sys.argv[1])
