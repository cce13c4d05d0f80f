"""Run the CPU oracle on the same workloads (test helper; oracle side only)."""
from __future__ import annotations

import concurrent.futures as cf
import multiprocessing as mp
import os

import numpy as np

from oracle import mdlstm


def _one(args):
    x, p64, dy, backward = args
    Y, cache = mdlstm.layer_forward(x, *p64)
    if not backward:
        return Y, None
    return Y, mdlstm.layer_backward(cache, dy, *p64)


def default_workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def run_layer(xs, params, dys, backward=True, workers=1):
    """Per example, each computed alone: Y (and dX), plus weight gradients summed over examples."""
    p64 = [np.asarray(t, np.float64) for t in params]
    jobs = [(x, p64, (dys[k] if backward else None), backward) for k, x in enumerate(xs)]
    if workers > 1 and len(jobs) > 1:
        with cf.ProcessPoolExecutor(workers, mp_context=mp.get_context("fork")) as ex:
            results = list(ex.map(_one, jobs))
    else:
        results = [_one(j) for j in jobs]
    out = {"Y": [r[0] for r in results], "dX": []}
    if backward:
        H = params[1].shape[2] // 2
        C = params[0].shape[2]
        acc = [np.zeros((4, 5 * H, C)), np.zeros((4, 5 * H, 2 * H)), np.zeros((4, 5 * H))]
        for _, g in results:
            dX, dWx, dU, db = g
            out["dX"].append(dX)
            acc = [a + b for a, b in zip(acc, (dWx, dU, db))]
        out["dWx"], out["dU"], out["db"] = acc
    return out
