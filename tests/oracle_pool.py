"""Runs the fp64 oracle over many units in parallel worker processes (test
infrastructure: the full-size parity checks score every unit of a batch).

Workers are started with the "spawn" method, so they are fresh interpreters
that never touch the GPU; each runs NumPy with one BLAS thread. A unit's
window queries, keys and values are sent as their raw storage (bf16 bit
patterns, or fp32) and widened exactly to fp64 in the worker, which returns
the oracle's fp32-rounded scores and its kept indices.
"""

from __future__ import annotations

import multiprocessing as mp
import os
from collections import deque

import numpy as np


def _widen(raw: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return (raw.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return raw.astype(np.float64)


def _init_worker():
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)


def _score(task):
    from oracle import jacap_oracle as jo
    key, dtype, q, k, v, budgets, kw = task
    o = jo.score_unit(_widen(q, dtype), _widen(k, dtype), _widen(v, dtype), **kw)
    s32 = jo.to_fp32(o["scores"])
    idx = {b: jo.select_top(s32, b) for b in budgets}
    return key, s32, idx, bool(o["singular"])


def workers() -> int:
    n = os.cpu_count() or 1
    return max(1, min(16, n))


def _raw(t):
    import torch
    t = t.detach()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def oracle_all_units(case, budgets=(), max_in_flight=None, **kw):
    """Yields (b, l, h, scores32, {budget: idx}, singular) for every unit of
    `case` (in completion order), running the oracle's score_unit with the
    keyword arguments `kw` (tau, ridge, cov_mode)."""
    w = case.workload
    g = w.num_q_heads // w.num_kv_heads
    dtype = w.dtype
    units = [(b, l, h) for b in range(case.num_seqs) for l in range(w.num_layers)
             for h in range(w.num_kv_heads)]
    nw = workers()
    cap = max_in_flight or 2 * nw
    ctx = mp.get_context("spawn")
    offs = np.concatenate([[0], np.cumsum(case.seq_lens)]).astype(np.int64)
    with ctx.Pool(nw, initializer=_init_worker) as pool:
        pending = deque()
        it = iter(units)
        done = False
        while True:
            while not done and len(pending) < cap:
                try:
                    b, l, h = next(it)
                except StopIteration:
                    done = True
                    break
                lo, hi = int(offs[b]), int(offs[b + 1])
                task = ((b, l, h), dtype, _raw(case.q_win[b, l, h * g:(h + 1) * g]),
                        _raw(case.k[l, h, lo:hi]), _raw(case.v[l, h, lo:hi]),
                        tuple(budgets), kw)
                pending.append(pool.apply_async(_score, (task,)))
            if not pending:
                break
            key, s32, idx, singular = pending.popleft().get()
            yield (*key, s32, idx, singular)
