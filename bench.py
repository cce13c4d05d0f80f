"""Benchmark of the packed four-direction MDLSTM layer on one MI355X.

Workload (default): the word-shaped batch — 256 examples of height 16 with
lognormal widths (median 40, clipped to [8, 200]), C_in 16, hidden 16, fp32,
packed into rows of width 1024; one step = forward + backward of the layer
over the whole batch. The same batch is also run last-minute padded (every
example padded to the batch maximum) for the packed-vs-padded speed-up.

Metric: useful cell-updates/s = 4 directions x sum(h*w) / step time, the same
useful count for both layouts. Inputs are resident in HBM before timing.

Prints one JSON line. Options: --gpus N (only 1 is supported), --steps K,
--warmup W, --config {1,2,3,5}, --no-cpu, --no-padded.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, GB/s
PEAK_FP32_MFMA_TFLOPS = 157.3  # dense fp32 matrix
PEAK_BF16_MFMA_TFLOPS = 2500.0  # dense bf16 matrix

PHASES = [("projection", 0, 1), ("zero_invalid", 1, 2), ("wavefront_fwd", 2, 3), ("wavefront_bwd", 4, 5),
          ("input_grad", 5, 6), ("weight_grad", 6, 7)]


def _parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 5])
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-padded", action="store_true", help="skip the padded-layout comparison")
    return ap.parse_args()


def algorithmic(wl, n_cells: int, unit_cells: int):
    """Algorithmic bytes and flops per launch of each kernel.

    unit_cells: cells covered by the scheduling rectangles (x4 directions below).
    n_cells: canvas cells (the dense GEMMs run over the whole canvas).
    """
    H, C = wl.hidden, wl.c_in
    s = 2 if wl.dtype == "bf16" else 4
    cd = 4 * unit_cells
    return {
        "projection": (n_cells * (C + 20 * H) * s + 20 * H * (C + 1) * s, 2.0 * n_cells * C * 20 * H),
        "zero_invalid": (0, 0.0),
        "wavefront_fwd": (cd * (10 * H * s + H * s + 4 * H), cd * 20.0 * H * H),
        "wavefront_bwd": (cd * (11 * H * s + 4 * H), cd * 20.0 * H * H),
        "input_grad": (n_cells * (20 * H + C) * s, 2.0 * n_cells * 20 * H * C),
        "weight_grad": (n_cells * (20 * H + C + 8 * H) * s, 2.0 * n_cells * 20 * H * (C + 2 * H + 1)),
    }


class Run:
    """One layout (packed or padded) of the workload, resident on the GPU."""

    def __init__(self, wl, kind: str):
        import torch

        from paper_1902_11208_amd import api

        self.torch, self.api = torch, api
        dev = "cuda"
        tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32

        def to_dev(a):
            return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(tdt).to(dev)

        torch.cuda.synchronize()
        t0 = time.perf_counter()
        if kind == "packed":
            units, ch, mask = api.pack_layout(wl.heights, wl.widths, wl.canvas_w)
            place, cw = units, wl.canvas_w
        else:
            units, place, ch, cw, mask = api.pad_layout(wl.heights, wl.widths)
        torch.cuda.synchronize()
        self.layout_ms = (time.perf_counter() - t0) * 1e3
        xs = [to_dev(x) for x in wl.examples()]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        self.x = api.pack_data(xs, place, ch, cw)
        torch.cuda.synchronize()
        self.scatter_ms = (time.perf_counter() - t0) * 1e3
        wx, u, b = (to_dev(p) for p in wl.params())
        self.dy = api.pack_data([to_dev(wl.dy(k)) for k in range(wl.n)], place, ch, cw)
        del xs
        self.layer = api.MDLSTMLayer(wx, u, b, ch, cw, units, mask)
        self.canvas_h, self.canvas_w = ch, cw
        self.n_cells = ch * cw
        self.unit_cells = int(np.sum(units[:, 2].astype(np.int64) * units[:, 3]))
        self.backward = not wl.forward_only

    def step(self):
        self.layer.forward(self.x)
        if self.backward:
            self.layer.backward(self.dy)

    def time(self, steps: int, warmup: int):
        torch = self.torch
        from paper_1902_11208_amd import _lib

        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(8)] for _ in range(steps)]
        for row in evs:  # create the underlying events
            for e in row:
                e.record()
        torch.cuda.synchronize()
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        L = _lib.lib()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        start.record()
        for k in range(steps):
            handles = (_lib.c_void * 8)(*[e.cuda_event for e in evs[k]])
            _lib.check(L.mdlstm_set_phase_events(8, handles))
            self.step()
        stop.record()
        torch.cuda.synchronize()
        wall_ms = (time.perf_counter() - t0) * 1e3
        _lib.check(L.mdlstm_set_phase_events(0, None))
        ev_ms = start.elapsed_time(stop)
        phase = {}
        for name, a, b in PHASES:
            if not self.backward and a >= 4:
                continue
            phase[name] = float(np.mean([evs[k][a].elapsed_time(evs[k][b]) for k in range(steps)]))
        return ev_ms / steps, wall_ms / steps, phase


def cpu_baseline(wl):
    """The oracle (float64 NumPy, each example alone) on the host cores."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle_run

    workers = oracle_run.default_workers()
    xs, params = wl.examples(), wl.params()
    dys = None if wl.forward_only else [wl.dy(k) for k in range(wl.n)]
    t0 = time.perf_counter()
    oracle_run.run_layer(xs, params, dys, backward=not wl.forward_only, workers=workers)
    dt = time.perf_counter() - t0
    useful = 4 * wl.useful_cells
    return {"value": useful / dt, "unit": "cell-updates/s", "cores": workers, "kind": "oracle",
            "sample": f"whole batch ({wl.n} examples, {useful} useful cell-directions), "
                      f"{'forward' if wl.forward_only else 'forward+backward'}, float64 NumPy, "
                      f"process pool of {workers} over examples, {dt:.1f} s wall"}


def main():
    args = _parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} (WORLD_SIZE {world}) is not supported; the layer has "
              "no multi-GPU path in this build (examples would be split across GPUs with an all-reduce of the "
              "weight gradients, see DESIGN.md)", file=sys.stderr)
        sys.exit(2)
    import torch

    from synth import configs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    from paper_1902_11208_amd import _lib

    if not os.path.exists(_lib.LIB_PATH):
        from paper_1902_11208_amd import build

        build.build()
    wl = configs.workload(args.config)
    useful = 4 * wl.useful_cells
    print(f"[bench] workload: {wl.name}, {wl.n} examples, useful cell-directions {useful}", file=sys.stderr,
          flush=True)

    packed = Run(wl, "packed")
    ms, wall_ms, phase = packed.time(args.steps, args.warmup)
    print(f"[bench] packed: {ms:.3f} ms/step (wall {wall_ms:.3f})", file=sys.stderr, flush=True)

    alg = algorithmic(wl, packed.n_cells, packed.unit_cells)
    phases_out = {}
    for name, t in phase.items():
        by, fl = alg[name]
        phases_out[name] = {"ms": round(t, 4), "GB_s": round(by / (t * 1e-3) / 1e9, 1) if t > 0 else None,
                            "TFLOP_s": round(fl / (t * 1e-3) / 1e12, 2) if t > 0 else None}
    dom = max(phase, key=lambda k: phase[k])
    by, fl = alg[dom]
    achieved = by / (phase[dom] * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None, "kernel": dom,
                "bytes_per_launch": int(by)}
    # the projection is a dense contraction: report its MFMA-peak fraction too
    proj_t = phase.get("projection")
    peak_mm = PEAK_BF16_MFMA_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS
    proj = None
    if proj_t:
        pf = alg["projection"][1] / (proj_t * 1e-3) / 1e12
        pb = alg["projection"][0] / (proj_t * 1e-3) / 1e9
        proj = {"TFLOP_s": round(pf, 2), "frac_mfma_peak": round(pf / peak_mm, 4), "GB_s": round(pb, 1),
                "frac_hbm_peak": round(pb / PEAK_HBM_GBS, 4)}

    padded = None
    if not args.no_padded:
        pr = Run(wl, "padded")
        pms, pwall, pphase = pr.time(max(3, args.steps // 2), args.warmup)
        padded = {"ms_per_step": round(pms, 4), "value": useful / (pms * 1e-3), "canvas_cells": pr.n_cells,
                  "unit_cells": pr.unit_cells, "speedup_packed_vs_padded": round(pms / ms, 3),
                  "phases_ms": {k: round(v, 4) for k, v in pphase.items()}}
        print(f"[bench] padded: {pms:.3f} ms/step", file=sys.stderr, flush=True)
        del pr

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(wl)
        print(f"[bench] cpu oracle: {cpu['value']:.3e} cell-updates/s on {cpu['cores']} cores", file=sys.stderr,
              flush=True)

    out = {
        "metric": "useful MDLSTM cell-updates/sec (4 dirs, fwd+bwd), packed vs padded; % roofline",
        "value": useful / (ms * 1e-3),
        "unit": "cell-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "examples": wl.n, "canvas": [packed.canvas_h, packed.canvas_w],
                   "useful_cell_dirs": useful, "forward_only": wl.forward_only},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "padded": padded,
        "projection": proj,
        "phases": phases_out,
        "layout_ms": round(packed.layout_ms, 3),
        "scatter_ms": round(packed.scatter_ms, 3),
        "wall_ms_per_step": round(wall_ms, 4),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
