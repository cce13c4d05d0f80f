"""Write the float64 oracle's full-batch weight gradients for the bf16 stress
batch (128 examples of height 48, widths 300-1200, C_in 64, H 128) to
``bf16_stress_grads.npz`` beside this script.

Test infrastructure: imports only the CPU oracle (``oracle/``) and the seeded
input generators (``synth/``). Every example is computed alone (Section V:
the packed result of each example equals its unpacked result), and the
gradients of L = sum(Y * dY) are summed over the examples in index order.
The oracle needs about an hour of core time for this batch, which is why its
result is stored instead of recomputed by the parity test.

Usage: python tests/golden/make_bf16_stress_grads.py [--workers N]
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import hashlib
import multiprocessing as mp
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import mdlstm  # noqa: E402
from synth import configs  # noqa: E402

OUT = os.path.join(HERE, "bf16_stress_grads.npz")


def input_digest(wl) -> str:
    """sha256 over the sizes and parameters the gradients depend on (examples
    and upstream gradients are keyed by the same seeds)."""
    h = hashlib.sha256()
    for a in (wl.heights, wl.widths, *wl.params()):
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def _one(k: int):
    wl = configs.workload(5)
    p64 = [np.asarray(t, np.float64) for t in wl.params()]
    _, cache = mdlstm.layer_forward(wl.example(k), *p64)
    _, dwx, du, db = mdlstm.layer_backward(cache, wl.dy(k), *p64)
    return k, dwx, du, db


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workers", type=int, default=max(1, len(os.sched_getaffinity(0))))
    args = ap.parse_args()
    wl = configs.workload(5)
    order = np.argsort(-wl.widths, kind="stable")  # longest first, to balance the pool
    parts = {}
    t0 = time.time()
    with cf.ProcessPoolExecutor(args.workers, mp_context=mp.get_context("fork")) as ex:
        for k, dwx, du, db in ex.map(_one, [int(k) for k in order]):
            parts[k] = (dwx, du, db)
            print(f"example {k} (width {wl.widths[k]}) done, {len(parts)}/{wl.n}, "
                  f"{time.time() - t0:.0f} s", flush=True)
    acc = [np.zeros_like(a) for a in parts[0]]
    for k in range(wl.n):
        acc = [a + b for a, b in zip(acc, parts[k])]
    np.savez_compressed(OUT, dWx=acc[0].astype(np.float32), dU=acc[1].astype(np.float32),
                        db=acc[2].astype(np.float32), inputs_sha256=np.array(input_digest(wl)))
    print(f"wrote {OUT}")


if __name__ == "__main__":
    main()
