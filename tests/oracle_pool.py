"""Runs the fp64 oracle's row_scores over many rows in a pool of worker processes.

Test infrastructure: the oracle itself is unchanged; this module only splits the
rows into chunks, hands each chunk to a worker that calls oracle.row_scores on it,
and stitches the per-row results back together in row order. Rows are
independent, so the result equals one row_scores call over all rows.

The weights are written once per call, in float64, to a file that every worker maps
read-only (the page cache holds one copy for all of them); each worker runs its BLAS
on one thread, so the pool spreads both the projections and the per-row sums over
the host cores. Workers are started with the "spawn" method: they are fresh
interpreters that never touch the GPU and import only numpy and the oracle.
"""
from __future__ import annotations

import atexit
import os
import shutil
import sys
import tempfile
import time
from concurrent.futures import ProcessPoolExecutor, as_completed

import numpy as np

_POOL = None
_POOL_N = 0
_W = {}   # worker side: path -> memory-mapped float64 weights


def _worker_init():
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:
        pass


def _weights(path):
    w = _W.get(path)
    if w is None:
        if len(_W) > 4:
            _W.clear()
        w = np.load(path, mmap_mode="r")
        _W[path] = w
    return w


def _task(args):
    (hs, ht, y, ws_path, wt_path, s_s, s_t, extras) = args
    ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    from oracle import olive_oracle as O
    ws = _weights(ws_path)
    wt = _weights(wt_path) if wt_path else None
    return O.row_scores(hs, ws, y, s_s, ht, wt, s_t, extras=extras)


def workers() -> int:
    """Worker count: the host cores, at most 16 (a shared host gives one GPU about 16)."""
    n = os.cpu_count() or 1
    try:
        n = min(n, len(os.sched_getaffinity(0)))
    except AttributeError:
        pass
    return max(1, min(16, n))


def _pool():
    global _POOL, _POOL_N
    if _POOL is None:
        import multiprocessing as mp
        _POOL_N = workers()
        _POOL = ProcessPoolExecutor(max_workers=_POOL_N, mp_context=mp.get_context("spawn"),
                                    initializer=_worker_init)
        atexit.register(shutdown)
    return _POOL


def shutdown():
    global _POOL
    if _POOL is not None:
        _POOL.shutdown(wait=True, cancel_futures=True)
        _POOL = None


def _scratch_dir(nbytes: int) -> str:
    """A directory with room for nbytes: /dev/shm when it has it, else the temp dir."""
    for d in ("/dev/shm", tempfile.gettempdir()):
        try:
            st = os.statvfs(d)
            if os.access(d, os.W_OK) and st.f_bavail * st.f_frsize > 1.5 * nbytes:
                return d
        except OSError:
            continue
    return tempfile.gettempdir()


def row_scores(hs, ws, y, s_s, ht=None, wt=None, s_t=1.0, extras=True, chunk=32,
               log=None):
    """oracle.row_scores(hs, ws, y, s_s, ht, wt, s_t, extras=extras), computed in chunks
    of rows by the worker pool. hs/ht: [n, d] host arrays; ws/wt: [d, V]."""
    n = len(y)
    if n == 0:
        from oracle import olive_oracle as O
        return O.row_scores(hs, ws, y, s_s, ht, wt, s_t, extras=extras)
    need = ws.shape[0] * ws.shape[1] * 8 + (0 if wt is None else wt.shape[0] * wt.shape[1] * 8)
    tmp = tempfile.mkdtemp(prefix="oracle_w_", dir=_scratch_dir(need))
    try:
        ws_path = os.path.join(tmp, "ws.npy")
        np.save(ws_path, np.asarray(ws, dtype=np.float64))
        wt_path = None
        if wt is not None:
            wt_path = os.path.join(tmp, "wt.npy")
            np.save(wt_path, np.asarray(wt, dtype=np.float64))
        pool = _pool()
        futs = {}
        for r0 in range(0, n, chunk):
            r1 = min(n, r0 + chunk)
            args = (np.asarray(hs[r0:r1], dtype=np.float64),
                    None if ht is None else np.asarray(ht[r0:r1], dtype=np.float64),
                    np.asarray(y[r0:r1]), ws_path, wt_path, s_s, s_t, extras)
            futs[pool.submit(_task, args)] = (r0, r1)
        parts = {}
        t0 = last = time.time()
        done = 0
        for f in as_completed(futs):
            r0, r1 = futs[f]
            parts[r0] = f.result()
            done += r1 - r0
            now = time.time()
            if log is not None and now - last > 10.0:
                log("oracle: %d/%d rows in %.0fs (%d workers)" % (done, n, now - t0, _POOL_N))
                last = now
        out = {}
        keys = parts[0].keys()
        for k in keys:
            out[k] = np.concatenate([parts[r0][k] for r0 in sorted(parts)], axis=0)
        return out
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
