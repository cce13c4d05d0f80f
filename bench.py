"""Benchmark of the packed four-direction MDLSTM layer on one MI355X.

Workload (default): the word-shaped batch — 256 examples of height 16 with
lognormal widths (median 40, clipped to [8, 200]), C_in 16, hidden 16, fp32,
packed into rows of width 1024; one step = forward + backward of the layer
over the whole batch. The same batch is also run last-minute padded (every
example padded to the batch maximum) for the packed-vs-padded speed-up.

Metric: useful cell-updates/s = 4 directions x sum(h*w) / step time, the same
useful count for both layouts. Inputs are resident in HBM before timing.

--config 4 times the three-layer stack on packed canvases instead (forward
+ backward of all layers and block convolutions; useful cells summed over
the layers). Per-step times are also given as median and minimum; the
packing time (placement + scatter) is reported separately and folded into
a second "with layout" rate.

Prints one JSON line. Options: --gpus N (only 1 is supported), --steps K,
--warmup W, --config {1,2,3,4,5}, --no-cpu, --no-padded.
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

COPY_BYTES = 256 << 20  # plain device copy used to calibrate FETCH_SIZE / WRITE_SIZE

PHASES = [("projection", 0, 1), ("zero_invalid", 1, 2), ("wavefront_fwd", 2, 3), ("wavefront_bwd", 4, 5),
          ("input_grad", 5, 6), ("weight_grad", 6, 7)]


def _parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-padded", action="store_true", help="skip the padded-layout comparison")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="finish with three plain 256 MiB device copies (reference for hardware byte counters)")
    return ap.parse_args()


def algorithmic(wl, n_cells: int, unit_cells: int, n_units: int = 0, cus: int = 256):
    """Algorithmic bytes and flops per launch of each kernel.

    unit_cells: cells covered by the scheduling rectangles (x4 directions below).
    n_cells: canvas cells (the dense GEMMs run over the whole canvas).
    n_units: units of the forward wavefront; with at least one per CU it also
    writes the zero output rows of the cells outside the rectangles.
    """
    H, C = wl.hidden, wl.c_in
    s = 2 if wl.dtype == "bf16" else 4
    cd = 4 * unit_cells
    zero = (n_cells - unit_cells) * 4 * H * s
    in_wave = n_units >= cus
    return {
        "projection": (n_cells * (C + 20 * H) * s + 20 * H * (C + 1) * s, 2.0 * n_cells * C * 20 * H),
        "zero_invalid": (0 if in_wave else zero, 0.0),
        "wavefront_fwd": (cd * (10 * H * s + H * s + 4 * H) + (zero if in_wave else 0), cd * 20.0 * H * H),
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

        xs = [to_dev(x) for x in wl.examples()]

        def layout():
            if kind == "packed":
                units, ch, mask = api.pack_layout(wl.heights, wl.widths, wl.canvas_w)
                return units, units, ch, wl.canvas_w, mask
            return api.pad_layout(wl.heights, wl.widths)

        # placement + mask, then the scatter of the examples: timed warm (median of 5)
        t_lay, t_sc = [], []
        for _ in range(6):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            units, place, ch, cw, mask = layout()
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            self.x = api.pack_data(xs, place, ch, cw)
            torch.cuda.synchronize()
            t_lay.append((t1 - t0) * 1e3)
            t_sc.append((time.perf_counter() - t1) * 1e3)
        self.layout_ms, self.scatter_ms = float(np.median(t_lay[1:])), float(np.median(t_sc[1:]))
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
        """Mean ms per step over the timed region, wall ms per step, per-phase
        ms and per-step ms.

        Recording an event costs the stream a few microseconds, so the timed
        region records only the step boundaries and the two boundaries of the
        dominant kernel (chosen from the last warm-up step, which records all
        eight); the full phase breakdown comes from a second pass of the same
        number of steps after it. The dominant kernel's duration in the
        returned phases is the one measured in the timed region.
        """
        torch = self.torch
        from paper_1902_11208_amd import _lib

        L = _lib.lib()
        phases = [(n, a, b) for n, a, b in PHASES if self.backward or b < 4]

        def events(n):
            evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
            for e in evs:  # create the underlying events
                e.record()
            return evs

        def handles(evs, keep=range(8)):
            return (_lib.c_void * 8)(*[evs[i].cuda_event if i in keep else None for i in range(8)])

        for _ in range(max(warmup - 1, 0)):
            self.step()
        last_warm = events(8)
        torch.cuda.synchronize()
        _lib.check(L.mdlstm_set_phase_events(8, handles(last_warm)))
        self.step()
        torch.cuda.synchronize()
        warm = {n: last_warm[a].elapsed_time(last_warm[b]) for n, a, b in phases}
        dom = max(warm, key=lambda k: warm[k])
        da, db = next((a, b) for n, a, b in phases if n == dom)

        marks = events(steps + 1)
        dev = [events(8) for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(steps):
            marks[k].record()
            _lib.check(L.mdlstm_set_phase_events(8, handles(dev[k], (da, db))))
            self.step()
        marks[steps].record()
        torch.cuda.synchronize()
        wall_ms = (time.perf_counter() - t0) * 1e3
        ev_ms = marks[0].elapsed_time(marks[steps])
        per_step = [marks[k].elapsed_time(marks[k + 1]) for k in range(steps)]
        dom_ms = float(np.mean([dev[k][da].elapsed_time(dev[k][db]) for k in range(steps)]))

        evs = [events(8) for _ in range(steps)]
        torch.cuda.synchronize()
        for k in range(steps):
            _lib.check(L.mdlstm_set_phase_events(8, handles(evs[k])))
            self.step()
        torch.cuda.synchronize()
        _lib.check(L.mdlstm_set_phase_events(0, None))
        phase = {n: float(np.mean([evs[k][a].elapsed_time(evs[k][b]) for k in range(steps)])) for n, a, b in phases}
        phase[dom] = dom_ms
        return ev_ms / steps, wall_ms / steps, phase, per_step

    def time_stepwise_forward(self, steps: int, warmup: int) -> float:
        """Mean forward-wavefront time when it runs as one launch per diagonal from a HIP graph."""
        torch = self.torch
        from paper_1902_11208_amd import _lib

        for _ in range(warmup):
            self.layer.forward_stepwise(self.x)
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(8)] for _ in range(steps)]
        for row in evs:
            for e in row:
                e.record()
        torch.cuda.synchronize()
        L = _lib.lib()
        for k in range(steps):
            _lib.check(L.mdlstm_set_phase_events(8, (_lib.c_void * 8)(*[e.cuda_event for e in evs[k]])))
            self.layer.forward_stepwise(self.x)
        torch.cuda.synchronize()
        _lib.check(L.mdlstm_set_phase_events(0, None))
        return float(np.mean([evs[k][2].elapsed_time(evs[k][3]) for k in range(steps)]))


class StackRun:
    """The three-layer stack (block reshape, MDLSTM layers, block convolutions) resident on the GPU."""

    def __init__(self, wl, kind: str):
        import torch

        from paper_1902_11208_amd import api, stack

        self.torch = torch
        dev = "cuda"

        def to_dev(a):
            return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)

        layers, convs = wl.params()
        dl = [tuple(to_dev(t) for t in p) for p in layers]
        dc = [tuple(to_dev(t) for t in p) for p in convs]
        imgs = [to_dev(wl.image(k)) for k in range(wl.n)]
        # layouts of all layers (+ buffers), then the block reshape of the images: timed warm (median of 3)
        t_lay, t_sc = [], []
        for _ in range(4):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            self.st = stack.MDLSTMStack(dl, dc, wl.heights, wl.widths, wl.canvas_w, block=wl.block, kind=kind)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            self.x = self.st.pack_input(imgs)
            torch.cuda.synchronize()
            t_lay.append((t1 - t0) * 1e3)
            t_sc.append((time.perf_counter() - t1) * 1e3)
        self.layout_ms, self.scatter_ms = float(np.median(t_lay[1:])), float(np.median(t_sc[1:]))
        ch, cw = self.st.canvas[-1]
        self.dy = api.pack_data([to_dev(wl.dy(k)) for k in range(wl.n)], self.st.rects[-1], ch, cw)
        self.canvas_h, self.canvas_w = self.st.canvas[0]
        self.n_cells = sum(h * w for h, w in self.st.canvas)
        self.unit_cells = sum(int(np.sum(l.prep.rects_np[:, 2].astype(np.int64) * l.prep.rects_np[:, 3]))
                              for l in self.st.layers)
        self.backward = True

    def step(self):
        self.st.forward(self.x)
        self.st.backward(self.dy)

    def time(self, steps: int, warmup: int):
        torch = self.torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        start.record()
        for k in range(steps):
            evs[k][0].record()
            self.step()
            evs[k][1].record()
        stop.record()
        torch.cuda.synchronize()
        wall_ms = (time.perf_counter() - t0) * 1e3
        per_step = [a.elapsed_time(b) for a, b in evs]
        return start.elapsed_time(stop) / steps, wall_ms / steps, {}, per_step


def cpu_baseline_stack(wl, max_images: int = 8):
    """The oracle on a bounded sample of the stack batch (each image alone, float64)."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle_run

    workers = oracle_run.default_workers()
    ks = list(range(min(max_images, wl.n)))
    layers, convs = wl.params()
    t0 = time.perf_counter()
    oracle_run.run_stack([wl.image(k) for k in ks], layers, convs, [wl.dy(k) for k in ks], wl.block,
                         workers=workers)
    dt = time.perf_counter() - t0
    useful = 0
    for k in ks:
        h, w = int(wl.heights[k]), int(wl.widths[k])
        useful += 4 * sum((h // wl.block[0] ** (l + 1)) * (w // wl.block[1] ** (l + 1)) for l in range(3))
    return {"value": useful / dt, "unit": "cell-updates/s", "cores": workers, "kind": "oracle",
            "sample": f"{len(ks)} of {wl.n} images, all three layers and convolutions, forward+backward, "
                      f"float64 NumPy, process pool of {workers} over images, {dt:.1f} s wall"}


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
              "no multi-GPU path (examples would be split across GPUs with an all-reduce of the weight "
              "gradients)", file=sys.stderr)
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
    if args.config == 4:
        wl = configs.stack_workload()
        wl.name, wl.dtype, wl.forward_only = ("line stack: 32 x h64 widths 400-1600, MDLSTM 16/32/64 with 2x4 "
                                              "block convolutions", "f32", False)
        RunCls = StackRun
    else:
        wl = configs.workload(args.config)
        RunCls = Run
    print(f"[bench] workload: {wl.name}, {wl.n} examples", file=sys.stderr, flush=True)

    packed = RunCls(wl, "packed")
    useful = 4 * packed.unit_cells
    ms, wall_ms, phase, per_step = packed.time(args.steps, args.warmup)
    print(f"[bench] packed: {ms:.3f} ms/step (wall {wall_ms:.3f}), useful cell-directions {useful}",
          file=sys.stderr, flush=True)
    pack_ms = packed.layout_ms + packed.scatter_ms

    if args.config == 4:
        roofline, proj, phases_out, stepwise = None, None, {}, None
    else:
        roofline, proj, phases_out = _rooflines(wl, packed, phase)
        stepwise = packed.time_stepwise_forward(max(3, args.steps // 2), args.warmup)
        print(f"[bench] forward wavefront, one launch per diagonal from a HIP graph: {stepwise:.3f} ms",
              file=sys.stderr, flush=True)

    padded = None
    if not args.no_padded:
        pr = RunCls(wl, "padded")
        pms, pwall, pphase, pper = pr.time(max(3, args.steps // 2), args.warmup)
        padded = {"ms_per_step": round(pms, 4), "median_ms": round(float(np.median(pper)), 4),
                  "value": useful / (pms * 1e-3), "canvas_cells": pr.n_cells,
                  "unit_cells": pr.unit_cells, "speedup_packed_vs_padded": round(pms / ms, 3),
                  "layout_ms": round(pr.layout_ms + pr.scatter_ms, 3),
                  "phases_ms": {k: round(v, 4) for k, v in pphase.items()}}
        print(f"[bench] padded: {pms:.3f} ms/step", file=sys.stderr, flush=True)
        del pr

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline_stack(wl) if args.config == 4 else cpu_baseline(wl)
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
        "wavefront_fwd_stepwise_graph_ms": None if stepwise is None else round(stepwise, 4),
        "median_ms": round(float(np.median(per_step)), 4),
        "min_ms": round(float(np.min(per_step)), 4),
        "layout_ms": round(packed.layout_ms, 3),
        "scatter_ms": round(packed.scatter_ms, 3),
        "value_with_layout": useful / ((ms + pack_ms) * 1e-3),
        "wall_ms_per_step": round(wall_ms, 4),
    }
    if args.copy_calibration:
        a = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
    print(json.dumps(out), flush=True)


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed hardware-counter summary,
    or None when there is none or the kernel source changed since it was taken."""
    import glob
    import hashlib

    for path in glob.glob(os.path.join(ROOT, "profiles", "traffic_*.md")):
        fields = {}
        for line in open(path):
            if ":" in line and not line.startswith(("|", "#", " ")):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
        if fields.get("kernel") != kernel or fields.get("workload") != workload:
            continue
        for k, v in fields.items():
            if k.startswith("source_sha256"):
                src = k[k.index("(") + 1:k.index(")")]
                digest = hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest()
                if digest == v:
                    return int(fields["traffic_bytes_per_launch"])
    return None


def _rooflines(wl, packed, phase):
    """Per-phase rates, the dominant kernel's HBM roofline and the projection's MFMA fraction."""
    import torch

    cus = torch.cuda.get_device_properties(0).multi_processor_count
    alg = algorithmic(wl, packed.n_cells, packed.unit_cells, 4 * len(wl.heights), cus)
    phases_out = {}
    for name, t in phase.items():
        by, fl = alg[name]
        phases_out[name] = {"ms": round(t, 4), "GB_s": round(by / (t * 1e-3) / 1e9, 1) if t > 0 else None,
                            "TFLOP_s": round(fl / (t * 1e-3) / 1e12, 2) if t > 0 else None}
    dom = max(phase, key=lambda k: phase[k])
    by, fl = alg[dom]
    achieved = by / (phase[dom] * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4),
                "traffic": measured_traffic(dom, "words") if wl.cid == 2 else None, "kernel": dom,
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
    return roofline, proj, phases_out


if __name__ == "__main__":
    main()
