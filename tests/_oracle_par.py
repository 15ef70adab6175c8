"""Oracle calls spread over the host's cores, for the full-size comparisons.

Test infrastructure only.  Each helper splits the samples into contiguous
chunks, runs the oracle on every chunk in its own thread (the oracle's C calls
release the interpreter lock) and combines the chunks in chunk order, so the
result does not depend on thread timing.  At most 16 threads.
"""
from __future__ import annotations

import os
import threading

import numpy as np

from oracle import oracle as orc


def cores() -> int:
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return max(1, min(n, 16))


def _chunks(n, k):
    k = max(1, min(k, n))
    bounds = [n * t // k for t in range(k + 1)]
    return [(bounds[t], bounds[t + 1]) for t in range(k)]


def _run(fn, ranges):
    out = [None] * len(ranges)
    err = []

    def work(t):
        try:
            out[t] = fn(*ranges[t])
        except BaseException as e:  # re-raised in the caller's thread
            err.append(e)

    threads = [threading.Thread(target=work, args=(t,)) for t in range(len(ranges))]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    if err:
        raise err[0]
    return out


def grad_sum(layers, params, x, y):
    """orc.grad_sum over all samples -> (G, per-sample losses, per-sample gaps);
    the chunk sums are added in chunk order (fp64)."""
    n = len(y)
    if n == 0:
        return np.zeros(orc.n_params(layers)), np.zeros(0), np.zeros(0)
    parts = _run(lambda a, b: orc.grad_sum(layers, params, x[a:b], y[a:b], with_gaps=True),
                 _chunks(n, cores()))
    g = np.zeros_like(parts[0][0])
    for q in parts:
        g += q[0]
    return g, np.concatenate([q[1] for q in parts]), np.concatenate([q[2] for q in parts])


def evaluate(layers, params, x, y):
    """orc.evaluate over all samples -> (outputs [n][n_out], wrong count)."""
    parts = _run(lambda a, b: orc.evaluate(layers, params, x[a:b], y[a:b]), _chunks(len(y), cores()))
    return np.concatenate([q[0] for q in parts]), sum(q[1] for q in parts)


def forward_backward(layers, params, x, y, idx, **kw):
    """orc.forward_backward for the samples idx -> list of result dicts, in idx order."""
    idx = list(idx)

    def chunk(a, b):
        return [orc.forward_backward(layers, params, x[i], int(y[i]), **kw) for i in idx[a:b]]

    parts = _run(chunk, _chunks(len(idx), cores())) if idx else []
    return [r for q in parts for r in q]
