"""Run the CPU fp64 oracle over many sequences at once, one process per core.

Test infrastructure: the full-size parity tests compare every output of a
decode step (and of the chunked prefill) with the oracle, and the oracle is
plain numpy that handles one sequence at a time, so the sequences (or slices of
a sequence's query rows) are spread over a pool of worker processes. Workers are started with ``spawn`` (never ``fork`` from a process
that has initialised the GPU) and import nothing but numpy and ``oracle``.

Jobs are self-contained one-sequence problems (the sequence's query rows, its
own blocks copied out of the cache, a block table renumbered to them): pure
data movement, prepared by the caller. No attention arithmetic lives here.
"""

from __future__ import annotations

import atexit
import multiprocessing as mp
import os
import time

_POOL = None
_CORES = 0
# Host cores that the process driving one MI355X may use (one GPU's share of
# an 8-GPU host); a pool larger than that only oversubscribes them.
MAX_CORES = 16


def cores_available() -> int:
    return len(os.sched_getaffinity(0))


def _worker_init():
    # one BLAS thread per worker: the pool already uses every core
    for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[k] = "1"


def _run(job):
    import oracle

    kind, key, kw = job
    fn = {"decode": oracle.paged_decode_attention,
          "multi_token": oracle.paged_multi_token_attention,
          "prefill": oracle.paged_prefill_attention}[kind]
    return key, fn(**kw)


def pool():
    """The shared worker pool (created on first use, closed at exit)."""
    global _POOL, _CORES
    if _POOL is None:
        _CORES = min(cores_available(), MAX_CORES)
        _POOL = mp.get_context("spawn").Pool(_CORES, initializer=_worker_init)
        atexit.register(close)
    return _POOL


def cores_used() -> int:
    return _CORES


def close():
    """Terminate the workers and wait for them (and the semaphore tracker
    that spawn starts) to exit, so no process outlives the caller."""
    global _POOL
    if _POOL is not None:
        _POOL.terminate()
        _POOL.join()
        _POOL = None
        try:
            from multiprocessing import resource_tracker
            resource_tracker._resource_tracker._stop()
        except Exception:  # the tracker API is private; a leftover tracker exits with the parent
            pass


def run_jobs(jobs, on_result, window=None, progress=None):
    """Run ``jobs`` (an iterable of (kind, key, kwargs)) through the pool,
    keeping at most ``window`` jobs in flight so that the parent never holds
    more than that many jobs' inputs; ``on_result(key, out)`` receives each
    result. ``progress(done, seconds)`` is called about every 10 s."""
    p = pool()
    window = window or 2 * _CORES
    pending = []
    done = 0
    t0 = last = time.perf_counter()
    it = iter(jobs)
    exhausted = False
    while pending or not exhausted:
        while not exhausted and len(pending) < window:
            try:
                job = next(it)
            except StopIteration:
                exhausted = True
                break
            pending.append(p.apply_async(_run, (job,)))
        if pending:
            key, out = pending.pop(0).get()
            on_result(key, out)
            done += 1
            now = time.perf_counter()
            if progress is not None and now - last > 10:
                progress(done, now - t0)
                last = now
    return time.perf_counter() - t0
