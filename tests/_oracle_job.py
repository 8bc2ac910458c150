"""Full fp64 oracle of a named workload, fanned out over host cores.

Test infrastructure.  A GPU test process has the device open, so it does not
fork worker processes itself: it starts this module as a fresh interpreter
(``python tests/_oracle_job.py <name> <out.npy>``), which rebuilds the same
seeded workload, evaluates the oracle on every output in forked worker
processes (one BLAS thread each) and saves the result.  This process never
imports torch or touches the GPU.

Every (sequence, kv head) pair of a one-query workload goes through
``oracle.attend_pairs``; the masked variants (several query tokens, sliding
window) go sequence by sequence through ``oracle.attend_masked``.  The result
has the shape of the workload's q: [B, Hq, D], or [B, Tq, Hq, D].
"""
from __future__ import annotations

import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

_JOB = None  # (workload, items), set before the workers fork


def host_workers(cap: int = 16) -> int:
    """Host threads this process may use, at most `cap` (one GPU's share)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(cap, n))


def _masked(w) -> bool:
    return w.num_queries > 1 or w.window > 0


def _work(chunk):
    import oracle
    from threadpoolctl import threadpool_limits
    w, _ = _JOB
    res = []
    with threadpool_limits(limits=1):
        for item in chunk:
            if _masked(w):
                b = item
                q4 = w.q if w.q.ndim == 4 else w.q[:, None]
                o, _ = oracle.attend_masked(q4[b:b + 1], w.k_cache, w.v_cache, w.block_table[b:b + 1],
                                            w.context_lens[b:b + 1], w.scale, w.window)
                res.append((b, o[0]))
            else:
                (o, _), = oracle.attend_pairs(w.q, w.k_cache, w.v_cache, w.block_table, w.context_lens,
                                              w.scale, [item]).values()
                res.append((item, o))
    return res


def full_reference(w, workers: int) -> np.ndarray:
    """The oracle on every output of workload `w`, in `workers` forked
    processes (1 = in this process)."""
    global _JOB
    g = w.num_q_heads // w.num_kv_heads
    if _masked(w):
        items = list(range(w.batch))
        cost = [int(w.context_lens[b]) for b in items]
    else:
        items = [(b, kv) for b in range(w.batch) for kv in range(w.num_kv_heads)]
        cost = [int(w.context_lens[b]) for b, _ in items]
    # longest first, dealt round-robin: balanced chunks, many per worker
    order = sorted(range(len(items)), key=lambda i: -cost[i])
    nchunks = max(1, min(len(items), 8 * workers))
    chunks = [[items[i] for i in order[j::nchunks]] for j in range(nchunks)]
    _JOB = (w, items)
    try:
        if workers == 1:
            parts = [_work(c) for c in chunks]
        else:
            import multiprocessing as mp
            with mp.get_context("fork").Pool(workers) as pool:
                parts = pool.map(_work, chunks, chunksize=1)
    finally:
        _JOB = None
    out = np.zeros(w.q.shape, dtype=np.float64)
    for part in parts:
        for item, o in part:
            if _masked(w):
                out[item] = o.reshape(out[item].shape)
            else:
                b, kv = item
                out[b, ..., kv * g:(kv + 1) * g, :] = o
    return out


class Job:
    """A running oracle job for a named workload (see :func:`start`)."""

    def __init__(self, name: str, path: str, proc: subprocess.Popen):
        self.name, self.path, self.proc = name, path, proc

    def result(self, timeout: float = 600.0) -> np.ndarray:
        try:
            rc = self.proc.wait(timeout=timeout)
        except subprocess.TimeoutExpired:
            self.proc.kill()
            self.proc.wait()
            raise
        log = self.proc.stdout.read() if self.proc.stdout else ""
        if rc != 0:
            raise RuntimeError(f"oracle job for {self.name} failed (rc {rc}):\n{log}")
        sys.stdout.write(log)
        sys.stdout.flush()
        try:
            return np.load(self.path)
        finally:
            os.unlink(self.path)


def start(name: str, tmpdir: str, workers: int = 0) -> Job:
    """Start the full oracle of workload `name` in a fresh interpreter."""
    path = os.path.join(tmpdir, f"oracle_{name}.npy")
    cmd = [sys.executable, "-u", os.path.abspath(__file__), name, path, str(workers or host_workers())]
    proc = subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, cwd=ROOT)
    return Job(name, path, proc)


def main(argv):
    import workloads as W
    name, path, workers = argv[0], argv[1], int(argv[2])
    t0 = time.perf_counter()
    w = W.make(name)
    t1 = time.perf_counter()
    out = full_reference(w, workers)
    t2 = time.perf_counter()
    np.save(path, out)
    print(f"oracle job {name}: generated in {t1 - t0:.1f} s, {out.size} outputs in {t2 - t1:.1f} s "
          f"on {workers} processes", flush=True)


if __name__ == "__main__":
    main(sys.argv[1:])
