"""Runs the float64 oracle over large token counts in parallel threads.

Only orchestration: every number comes from an `oracle.duo_ref` function
called on a contiguous range of tokens.  Stage-1 terms and the layer
objective are sums over tokens, so the ranges' results add up exactly to the
single call's (up to the order of the float64 additions).  numpy releases the
GIL in its sorts and BLAS calls; the BLAS threads are limited so that the
workers together use the host's cores once.
"""

from __future__ import annotations

import os
from concurrent.futures import FIRST_COMPLETED, ThreadPoolExecutor, wait

from oracle import duo_ref as R

try:
    from threadpoolctl import threadpool_limits
except ImportError:  # pragma: no cover
    threadpool_limits = None


def host_cores() -> int:
    n = len(os.sched_getaffinity(0))
    cap = int(os.environ.get("OMP_NUM_THREADS", n) or n)
    return max(1, min(n, cap))


def _ranges(m, parts):
    step = -(-m // parts)
    step = -(-step // 8192) * 8192          # whole oracle token chunks
    return [(t0, min(m, t0 + step)) for t0 in range(0, m, step)]


def _reduce(fn, add, m, workers=None, label="oracle"):
    """fn(t0, t1) over token ranges (four per worker) in parallel threads;
    results are folded with add(acc, part) as they finish, so at most
    `workers` partial results are alive; one progress line per range."""
    workers = workers or min(8, host_cores())
    blas = max(1, host_cores() // workers)
    ranges = _ranges(m, 4 * workers)
    acc = None
    ctx = threadpool_limits(limits=blas) if threadpool_limits is not None else None
    if ctx is not None:
        ctx.__enter__()
    try:
        with ThreadPoolExecutor(workers) as ex:
            todo = list(reversed(ranges))
            pending = set()
            done_n = 0
            while todo or pending:
                while todo and len(pending) < workers:
                    pending.add(ex.submit(fn, *todo.pop()))
                done, pending = wait(pending, return_when=FIRST_COMPLETED)
                for f in done:
                    part = f.result()
                    acc = part if acc is None else add(acc, part)
                    done_n += 1
                    print(f"[oracle] {label}: {done_n}/{len(ranges)} token ranges", flush=True)
                del done, f, part
    finally:
        if ctx is not None:
            ctx.__exit__(None, None, None)
    return acc


def _add_terms(acc, part):
    for x, y in zip(acc, part):
        x += y
    return acc


def hessian_terms(X_src, p_x, X_dense=None, workers=None):
    """R.hessian_terms over all tokens, token ranges in parallel."""
    return _reduce(lambda t0, t1: R.hessian_terms(X_src[t0:t1], p_x, None if X_dense is None else X_dense[t0:t1]),
                   _add_terms, X_src.shape[0], workers, "stage 1")


def hessian_entries(X_src, p_x, idx, X_dense=None, workers=None, rows=None):
    """R.hessian_entries over all tokens, token ranges in parallel."""
    def add(acc, part):
        for key in acc:
            acc[key] += part[key]
        return acc
    return _reduce(lambda t0, t1: R.hessian_entries(X_src, p_x, idx, X_dense=X_dense, t0=t0, t1=t1, rows=rows),
                   add, X_src.shape[0], workers, "stage-1 entries")


def objectives(W, W_hats, X_src, p_x, X_dense=None, workers=None):
    """R.objective of each candidate in W_hats over all tokens."""
    return _reduce(lambda t0, t1: R.objective(W, list(W_hats), X_src[t0:t1], p_x,
                                              None if X_dense is None else X_dense[t0:t1]),
                   lambda acc, part: [x + y for x, y in zip(acc, part)], X_src.shape[0], workers, "objective")
