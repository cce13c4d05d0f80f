"""Run the CPU oracle on the same workloads (test helper; oracle side only)."""
from __future__ import annotations

import concurrent.futures as cf
import multiprocessing as mp
import os

import numpy as np

from oracle import mdlstm


def _one(args):
    x, p64, dy, backward = args
    v = p64[3] if len(p64) > 3 else None
    Y, cache = mdlstm.layer_forward(x, *p64[:3], v=v)
    if not backward:
        return Y, None
    return Y, mdlstm.layer_backward(cache, dy, *p64[:3], v=v)


def default_workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


_LIMITS = None


def single_threaded_blas():
    """Hold NumPy's BLAS to one thread in this process (pool workers each use one core)."""
    global _LIMITS
    from threadpoolctl import threadpool_limits

    _LIMITS = threadpool_limits(limits=1)


def _pool_map(fn, jobs, workers, progress):
    """fn over jobs in a fork pool (one BLAS thread per worker), results in job
    order; with `progress`, a line per finished job (long oracle runs stay
    visibly alive)."""
    if workers <= 1 or len(jobs) <= 1:
        out = []
        for i, j in enumerate(jobs):
            out.append(fn(j))
            if progress:
                print(f"{progress}: {i + 1}/{len(jobs)} done", flush=True)
        return out
    results = [None] * len(jobs)
    with cf.ProcessPoolExecutor(workers, mp_context=mp.get_context("fork"), initializer=single_threaded_blas) as ex:
        futs = {ex.submit(fn, j): i for i, j in enumerate(jobs)}
        for done, f in enumerate(cf.as_completed(futs), 1):
            results[futs[f]] = f.result()
            if progress:
                print(f"{progress}: job {futs[f]} finished, {done}/{len(jobs)}", flush=True)
    return results


def run_layer(xs, params, dys, backward=True, workers=1, progress=None):
    """Per example, each computed alone: Y (and dX), plus weight gradients summed
    over examples. params: (wx, u, b), or (wx, u, b, v) with memory-state
    matrices (then dV is summed too)."""
    p64 = [np.asarray(t, np.float64) for t in params]
    jobs = [(x, p64, (dys[k] if backward else None), backward) for k, x in enumerate(xs)]
    results = _pool_map(_one, jobs, workers, progress)
    out = {"Y": [r[0] for r in results], "dX": []}
    if backward:
        H = params[1].shape[2] // 2
        C = params[0].shape[2]
        acc = [np.zeros((4, 5 * H, C)), np.zeros((4, 5 * H, 2 * H)), np.zeros((4, 5 * H))]
        if len(params) > 3:
            acc.append(np.zeros((4, 3 * H, 2 * H)))
        for _, g in results:
            out["dX"].append(g[0])
            acc = [a + b for a, b in zip(acc, g[1:])]
        out["dWx"], out["dU"], out["db"] = acc[:3]
        if len(params) > 3:
            out["dV"] = acc[3]
    return out


def _stack_one(args):
    from oracle import stack

    image, layers, convs, dy3, block = args
    Y3, cache = stack.stack_forward(image, layers, convs, block)
    lg, cg, g = stack.stack_backward(cache, dy3, layers, convs, block)
    return Y3, lg, cg, g


def run_stack(images, layers, convs, dys, block=(2, 4), workers=1, progress=None):
    """Per image, alone: last output Y3, input-block gradient, and the summed layer/conv gradients."""
    l64 = [tuple(np.asarray(t, np.float64) for t in p) for p in layers]
    c64 = [tuple(np.asarray(t, np.float64) for t in p) for p in convs]
    jobs = [(np.asarray(im, np.float64), l64, c64, dys[k], block) for k, im in enumerate(images)]
    results = _pool_map(_stack_one, jobs, workers, progress)
    out = {"Y": [r[0] for r in results], "dX0": [r[3] for r in results]}
    lsum = [[np.zeros_like(a) for a in results[0][1][i]] for i in range(len(layers))]
    csum = [[np.zeros_like(a) for a in results[0][2][i]] for i in range(len(convs))]
    for _, lg, cg, _ in results:
        for i in range(len(layers)):
            lsum[i] = [a + b for a, b in zip(lsum[i], lg[i])]
        for i in range(len(convs)):
            csum[i] = [a + b for a, b in zip(csum[i], cg[i])]
    out["layer_grads"], out["conv_grads"] = lsum, csum
    return out


def _step_one(args):
    from oracle import head

    x, p64, w64, b64, label = args
    Y, cache = mdlstm.layer_forward(x, *p64)
    loss, dY, dW, db, logits, dlogits = head.head_loss_forward_backward(Y, w64, b64, label)
    g = mdlstm.layer_backward(cache, dY, *p64)
    return loss, logits, dlogits, dW, db, g


def run_training_step(xs, params, head_params, labels, workers=1, progress=None):
    """One training step per example, each alone: MDLSTM layer, the shared
    output layer with the row collapse, CTC loss, and back. Returns losses,
    logits, dlogits and dX per example, and every weight gradient summed."""
    p64 = [np.asarray(t, np.float64) for t in params]
    w64, b64 = (np.asarray(t, np.float64) for t in head_params)
    jobs = [(x, p64, w64, b64, labels[k]) for k, x in enumerate(xs)]
    results = _pool_map(_step_one, jobs, workers, progress)
    out = {"loss": np.array([r[0] for r in results]), "logits": [r[1] for r in results],
           "dlogits": [r[2] for r in results], "dX": [r[5][0] for r in results]}
    out["dWfc"] = sum(r[3] for r in results)
    out["dbfc"] = sum(r[4] for r in results)
    for i, nm in enumerate(("dWx", "dU", "db")):
        acc = np.zeros_like(results[0][5][i + 1])
        for r in results:
            acc = acc + r[5][i + 1]
        out[nm] = acc
    return out
