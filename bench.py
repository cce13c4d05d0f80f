"""Benchmark of the packed four-direction MDLSTM layer on one MI355X.

Headline workload: the line-shaped batch, the largest single-layer fp32
workload: 64 examples of height 32 with widths uniform in [200, 600], C_in 32,
hidden 32, fp32, packed into rows of width 2048. One step is the forward and
backward pass of the layer over the whole batch: projection, forward
wavefront, backward wavefront, input and weight gradients. The same batch is
also run last-minute padded (every example padded to the batch maximum,
Section VI-B) for the packed-vs-padded speed-up.

Metric: useful cell-updates/s = 4 directions x sum(h*w) / step time, with the
same useful count for both layouts. Inputs are resident in HBM before timing.

The other four workloads are measured the same way and nested under
"configs": the tiny forward-only batch, the word batch, the three-layer
stack (forward + backward of all layers and block convolutions, useful cells
summed over the layers) and the bf16 stress batch. Every workload carries
per-kernel times, the dominant kernel's roofline (algorithmic bytes and flops
per useful cell-direction, from the cost model of the method: projection
C_in*s/4 + 5H*s bytes and 10*C_in*H flops; forward wavefront 5H*s + H*s + 4H
bytes and 20H^2 flops; backward wavefront 11H*s + 4H bytes and 20H^2 flops;
gradients 6H*s + C_in*s/2 bytes and 20H^2 + 20*C_in*H flops; s = storage
bytes), the projection's MFMA fraction, the padded comparison and the CPU
oracle on the host cores (all cores and one core, timed before the GPU is
touched). The paper's own speed-ups are quoted as context.

Prints one JSON line. Options: --gpus N (only 1 is supported), --steps K,
--warmup W, --config {1,2,3,4,5} (headline workload; default 3), --no-nested,
--no-cpu, --no-padded.
"""
from __future__ import annotations

import argparse
import json
import multiprocessing as mp
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0           # MI355X HBM3E, GB/s
PEAK_FP32_MFMA_TFLOPS = 157.3   # dense fp32 matrix
PEAK_BF16_MFMA_TFLOPS = 2500.0  # dense bf16 matrix

COPY_BYTES = 256 << 20  # plain device copy used to calibrate FETCH_SIZE / WRITE_SIZE

METRIC = "useful MDLSTM cell-updates/sec (4 dirs, fwd+bwd), packed vs padded; % roofline"
HEADLINE = 3
NESTED = [1, 2, 4, 5]

# The paper's only speed figures: whole IAM training epochs, example packing
# against last-minute batch padding, each at the largest batch that fit.
PAPER_CONTEXT = {
    "source": "Table IV (IAM training epochs, example-packing vs last-minute batch padding)",
    "hardware": "two NVIDIA GeForce GTX 1080 cards, as the paper states",
    "words_speedup_packed_vs_padded": 6.6,
    "lines_speedup_packed_vs_padded": 1.46,
    "note": "whole-model epochs at batch 200 vs 20 (words) and 12 vs 8 (lines); the words gain is mostly the "
            "larger batch that fits in 11 GB once padding is gone, not per-cell speed",
}

# phase name -> (start event, end event) of mdlstm_set_phase_events
PHASES_FWD = [("projection", 0, 1), ("zero_invalid", 1, 2), ("wavefront_fwd", 2, 3)]
PHASES_FUSED = [("wavefront_bwd", 4, 5), ("gradients", 6, 7)]
PHASES_SPLIT = [("wavefront_bwd", 4, 5), ("input_grad", 5, 6), ("weight_grad", 6, 7)]


def _parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=HEADLINE, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--no-nested", action="store_true", help="measure the headline workload only")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baselines")
    ap.add_argument("--no-padded", action="store_true", help="skip the padded-layout comparisons")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="finish with three plain 256 MiB device copies (reference for hardware byte counters)")
    return ap.parse_args()


# ---------------------------------------------------------------------------
# Cost model (algorithmic work per useful cell-direction)
# ---------------------------------------------------------------------------
def algorithmic(H: int, C: int, s: int, useful_cells: int):
    """Bytes and flops per launch of each phase, counted over useful cells only
    (4 directions each): what the computation must move and do, whatever the
    kernels' layout. Gradient phases: fused (one kernel reading dZ once) or split."""
    cd = 4 * useful_cells
    return {
        "projection": (cd * (C * s / 4 + 5 * H * s), cd * 10.0 * C * H),
        "zero_invalid": (0.0, 0.0),
        "wavefront_fwd": (cd * (5 * H * s + H * s + 4 * H), cd * 20.0 * H * H),
        "wavefront_bwd": (cd * (H * s + 5 * H * s + 4 * H + 5 * H * s), cd * 20.0 * H * H),
        "gradients": (cd * (5 * H * s + C * s / 4 + H * s + C * s / 4), cd * (20.0 * H * H + 20.0 * C * H)),
        "input_grad": (cd * (5 * H * s + C * s / 4), cd * 10.0 * C * H),
        "weight_grad": (cd * (5 * H * s + C * s / 4 + H * s), cd * (20.0 * H * H + 10.0 * C * H)),
    }


def design_bytes(H: int, C: int, s: int, useful_cells: int, canvas_cells: int, unit_cells: int):
    """HBM bytes the kernels move beyond the cost model, by design: the
    projection over separator and padding cells (an upper bound: its waves
    skip 64-cell chunks without a rectangle cell), the activated gates the
    forward writes back for the backward, and the zero output rows."""
    cd = 4 * useful_cells
    return {
        "projection_non_useful_cells": (canvas_cells - useful_cells) * (C + 20 * H) * s,
        "wavefront_fwd_gate_writeback": cd * 5 * H * s,
        "wavefront_fwd_unit_padding_cells": 4 * (unit_cells - useful_cells) * (11 * H * s + 4 * H),
        "zero_invalid_rows": (canvas_cells - useful_cells) * 4 * H * s,
    }


def mfma_peak(dtype: str) -> float:
    return PEAK_BF16_MFMA_TFLOPS if dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS


def roofline(name: str, ms: float, by: float, fl: float, dtype: str, traffic=None):
    """The binding roofline of a kernel (whichever of HBM time and MFMA time
    its algorithmic work needs more of), its achieved rate against that peak,
    and the other one's fraction."""
    t = ms * 1e-3
    gbs, tfs = by / t / 1e9, fl / t / 1e12
    pk = mfma_peak(dtype)
    hbm_bound = by / (PEAK_HBM_GBS * 1e9) >= fl / (pk * 1e12)
    if hbm_bound:
        out = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
               "frac": round(gbs / PEAK_HBM_GBS, 4)}
    else:
        out = {"bound": "mfma", "achieved": round(tfs, 2), "peak": pk, "unit": "TFLOP/s",
               "frac": round(tfs / pk, 4)}
    out.update({"traffic": traffic, "kernel": name, "ms": round(ms, 4), "bytes_per_launch": int(by),
                "flops_per_launch": int(fl), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4),
                "frac_mfma": round(tfs / pk, 4)})
    return out


def phase_rates(phase_ms: dict, alg: dict, dtype: str, where: str):
    """Per-phase rates; a rate above a peak means the timing or the cost model is wrong."""
    out = {}
    for name, ms in phase_ms.items():
        by, fl = alg[name]
        gbs = by / (ms * 1e-3) / 1e9 if ms > 0 else None
        tfs = fl / (ms * 1e-3) / 1e12 if ms > 0 else None
        if (gbs and gbs > PEAK_HBM_GBS) or (tfs and tfs > mfma_peak(dtype)):
            raise SystemExit(f"bench.py: {where} phase {name} at {gbs:.0f} GB/s, {tfs:.1f} TFLOP/s exceeds the "
                             f"peak ({ms:.4f} ms for {by:.3g} B, {fl:.3g} flop)")
        out[name] = {"ms": round(ms, 4), "GB_s": None if gbs is None else round(gbs, 1),
                     "TFLOP_s": None if tfs is None else round(tfs, 2)}
    return out


def projection_fractions(ms: float, by: float, fl: float, dtype: str):
    t = ms * 1e-3
    tfs, gbs = fl / t / 1e12, by / t / 1e9
    pk = mfma_peak(dtype)
    attainable = min(pk, (fl / by) * PEAK_HBM_GBS / 1e3)  # TFLOP/s at its intensity
    return {"TFLOP_s": round(tfs, 2), "frac_mfma_peak": round(tfs / pk, 4), "GB_s": round(gbs, 1),
            "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 4), "attainable_TFLOP_s": round(attainable, 2),
            "frac_attainable": round(tfs / attainable, 4)}


# ---------------------------------------------------------------------------
# GPU runs
# ---------------------------------------------------------------------------
def _events(torch, n):
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
    for e in evs:  # create the underlying events
        e.record()
    return evs


def _handles(evs, keep=range(8)):
    from paper_1902_11208_amd import _lib

    return (_lib.c_void * 8)(*[evs[i].cuda_event if i in keep else None for i in range(8)])


class Run:
    """One layout (packed or padded) of a single-layer workload, resident on the GPU."""

    def __init__(self, wl, kind: str):
        import torch

        from paper_1902_11208_amd import api

        self.torch, self.api = torch, api
        dev = "cuda"
        tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32

        def to_dev(a):
            return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev).to(tdt)

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
        del xs
        wx, u, b = (to_dev(p) for p in wl.params())
        self.backward = not wl.forward_only
        if self.backward:
            self.dy = api.pack_data([to_dev(wl.dy(k)) for k in range(wl.n)], place, ch, cw)
        self.layer = api.MDLSTMLayer(wx, u, b, ch, cw, units, mask)
        self.canvas_h, self.canvas_w = ch, cw
        self.n_cells = ch * cw
        self.unit_cells = int(np.sum(units[:, 2].astype(np.int64) * units[:, 3]))
        fused = api.gradients_fused(wl.c_in, wl.hidden, api.dtype_code(tdt))
        self.phases = PHASES_FWD + ((PHASES_FUSED if fused else PHASES_SPLIT) if self.backward else [])

    def step(self):
        self.layer.forward(self.x)
        if self.backward:
            self.layer.backward(self.dy)

    def time(self, steps: int, warmup: int):
        """Mean ms per step over the timed region, wall ms per step, per-phase
        ms and per-step ms.

        Recording an event costs the stream a few microseconds, so the timed
        region records only the step boundaries and the two boundaries of the
        dominant kernel. A phase pass of the same number of steps before it
        records all eight boundaries: it gives the per-phase breakdown and
        picks the dominant kernel (the longest mean phase). The dominant
        kernel's duration in the returned phases is the one measured in the
        timed region.
        """
        torch = self.torch
        from paper_1902_11208_amd import _lib

        L = _lib.lib()
        for _ in range(warmup):
            self.step()

        evs = [_events(torch, 8) for _ in range(steps)]
        torch.cuda.synchronize()
        for k in range(steps):
            _lib.check(L.mdlstm_set_phase_events(8, _handles(evs[k])))
            self.step()
        torch.cuda.synchronize()
        phase = {n: float(np.mean([evs[k][a].elapsed_time(evs[k][b]) for k in range(steps)]))
                 for n, a, b in self.phases}
        dom = max(phase, key=lambda k: phase[k])
        da, db = next((a, b) for n, a, b in self.phases if n == dom)

        marks = _events(torch, steps + 1)
        dev = [_events(torch, 8) for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(steps):
            marks[k].record()
            _lib.check(L.mdlstm_set_phase_events(8, _handles(dev[k], (da, db))))
            self.step()
        marks[steps].record()
        torch.cuda.synchronize()
        wall_ms = (time.perf_counter() - t0) * 1e3
        _lib.check(L.mdlstm_set_phase_events(0, None))
        ev_ms = marks[0].elapsed_time(marks[steps])
        per_step = [marks[k].elapsed_time(marks[k + 1]) for k in range(steps)]
        phase[dom] = float(np.mean([dev[k][da].elapsed_time(dev[k][db]) for k in range(steps)]))
        return ev_ms / steps, wall_ms / steps, phase, per_step, dom

    def time_stepwise_forward(self, steps: int, warmup: int) -> float:
        """Mean forward-wavefront time when it runs as one launch per diagonal from a HIP graph."""
        torch = self.torch
        from paper_1902_11208_amd import _lib

        for _ in range(warmup):
            self.layer.forward_stepwise(self.x)
        evs = [_events(torch, 8) for _ in range(steps)]
        torch.cuda.synchronize()
        L = _lib.lib()
        for k in range(steps):
            _lib.check(L.mdlstm_set_phase_events(8, _handles(evs[k])))
            self.layer.forward_stepwise(self.x)
        torch.cuda.synchronize()
        _lib.check(L.mdlstm_set_phase_events(0, None))
        return float(np.mean([evs[k][2].elapsed_time(evs[k][3]) for k in range(steps)]))


class StackRun:
    """The three-layer stack (block reshape, MDLSTM layers, block convolutions) resident on the GPU."""

    def __init__(self, wl, kind: str):
        import torch

        from paper_1902_11208_amd import api, stack

        self.torch, self.api = torch, api
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
        self.layer_cells = [int(np.sum(l.prep.rects_np[:, 2].astype(np.int64) * l.prep.rects_np[:, 3]))
                            for l in self.st.layers]
        self.unit_cells = sum(self.layer_cells)
        self.layer_phases = []
        for l in self.st.layers:
            fused = api.gradients_fused(l.c_in, l.hidden, l.dtype)
            self.layer_phases.append(PHASES_FWD + (PHASES_FUSED if fused else PHASES_SPLIT))

    def step(self, layer_events=None, conv_events=None):
        """Forward and backward of the stack; with events, layer l's kernel
        boundaries go to layer_events[l] and convolution c's calls are
        bracketed by conv_events[c] = (fwd start, fwd end, bwd start, bwd end)."""
        from paper_1902_11208_amd import _lib

        L = _lib.lib()
        st = self.st

        def set_layer(li):
            if layer_events is not None:
                _lib.check(L.mdlstm_set_phase_events(8, _handles(layer_events[li])))

        x = self.x
        for li, layer in enumerate(st.layers):
            set_layer(li)
            y = layer.forward(x)
            if li < len(st.convs):
                if conv_events is not None:
                    conv_events[li][0].record()
                x = st.convs[li].forward(y)
                if conv_events is not None:
                    conv_events[li][1].record()
        g = self.dy
        for li in range(len(st.layers) - 1, -1, -1):
            set_layer(li)
            dx, _, _, _ = st.layers[li].backward(g)
            if li > 0:
                if conv_events is not None:
                    conv_events[li - 1][2].record()
                g, _, _ = st.convs[li - 1].backward(dx)
                if conv_events is not None:
                    conv_events[li - 1][3].record()
        if layer_events is not None:
            _lib.check(L.mdlstm_set_phase_events(0, None))

    def time(self, steps: int, warmup: int):
        """Mean ms per step (step boundaries only in the timed region), wall ms
        per step, per-kernel ms (layer l's phases as "L<l>.<phase>", the block
        convolutions as "conv<c>.fwd"/"conv<c>.bwd") from a second pass, per-step ms."""
        torch = self.torch
        for _ in range(warmup):
            self.step()
        marks = _events(torch, steps + 1)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(steps):
            marks[k].record()
            self.step()
        marks[steps].record()
        torch.cuda.synchronize()
        wall_ms = (time.perf_counter() - t0) * 1e3
        per_step = [marks[k].elapsed_time(marks[k + 1]) for k in range(steps)]
        runs = []
        for _ in range(steps):
            le = [_events(torch, 8) for _ in self.st.layers]
            ce = [_events(torch, 4) for _ in self.st.convs]
            torch.cuda.synchronize()
            self.step(le, ce)
            runs.append((le, ce))
        torch.cuda.synchronize()
        phase = {}
        for li, ph in enumerate(self.layer_phases):
            for n, a, b in ph:
                phase[f"L{li}.{n}"] = float(np.mean([r[0][li][a].elapsed_time(r[0][li][b]) for r in runs]))
        for ci in range(len(self.st.convs)):
            phase[f"conv{ci}.fwd"] = float(np.mean([r[1][ci][0].elapsed_time(r[1][ci][1]) for r in runs]))
            phase[f"conv{ci}.bwd"] = float(np.mean([r[1][ci][2].elapsed_time(r[1][ci][3]) for r in runs]))
        dom = max(phase, key=lambda k: phase[k])
        return marks[0].elapsed_time(marks[steps]) / steps, wall_ms / steps, phase, per_step, dom


def stack_algorithmic(wl, run):
    """Cost-model bytes and flops of every kernel of the stack step (per layer
    as for one layer; a block convolution reads its input block map and writes
    its output, 2*og*8H flops per output value, twice that backward)."""
    alg = {}
    bh, bw = wl.block
    for li, (H, C) in enumerate(zip(wl.hidden, wl.mdlstm_c_in)):
        for k, v in algorithmic(H, C, 4, run.layer_cells[li]).items():
            alg[f"L{li}.{k}"] = v
    for ci in range(len(run.st.convs)):
        H, og = wl.hidden[ci], wl.conv_out[ci] // 4
        out_cells = run.layer_cells[ci + 1]
        in_vals, out_vals = out_cells * bh * bw * 4 * H, out_cells * 4 * og
        flops = 2.0 * out_vals * bh * bw * H
        alg[f"conv{ci}.fwd"] = (4.0 * (in_vals + out_vals), flops)
        # backward: read input, output and its gradient; write the input gradient
        alg[f"conv{ci}.bwd"] = (4.0 * (2 * in_vals + 2 * out_vals), 2 * flops)
    return alg


def measure_gpu(cid: int, steps: int, warmup: int, padded: bool, stepwise: bool):
    """Every GPU figure of one workload; returns its result object."""
    from synth import configs

    if cid == 4:
        wl = configs.stack_workload()
        name = ("line stack: 32 x h64 widths 400-1600 (multiples of 64), 2x4 blocks, MDLSTM 16/32/64 with 2x4 "
                "block convolutions to 32 and 64 channels")
        dtype = "f32"
        RunCls = StackRun
    else:
        wl = configs.workload(cid)
        name, dtype = wl.name, ("bf16" if wl.dtype == "bf16" else "f32")
        RunCls = Run
    print(f"[bench] workload {cid}: {name}, {wl.n} examples", file=sys.stderr, flush=True)
    import torch

    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats()
    run = RunCls(wl, "packed")
    ms, wall_ms, phase, per_step, dom = run.time(steps, warmup)
    peak_mb = torch.cuda.max_memory_allocated() / 2**20
    if cid == 4:
        useful = 4 * run.unit_cells
        alg = stack_algorithmic(wl, run)
        forward_only = False
        layer_of = {f"L{li}": (H, C) for li, (H, C) in enumerate(zip(wl.hidden, wl.mdlstm_c_in))}
        proj_name = max((k for k in phase if k.endswith(".projection")), key=lambda k: phase[k])
        extra = {"layers": [{"hidden": H, "c_in": C, "useful_cell_dirs": 4 * u, "canvas": list(cv)}
                            for H, C, u, cv in zip(wl.hidden, wl.mdlstm_c_in, run.layer_cells, run.st.canvas)]}
        crit = max(int(h) + int(w) - 1 for h, w in zip(wl.heights // 2, wl.widths // 4))
    else:
        useful = 4 * wl.useful_cells
        alg = algorithmic(wl.hidden, wl.c_in, 2 if dtype == "bf16" else 4, wl.useful_cells)
        forward_only = wl.forward_only
        proj_name = "projection"
        s = 2 if dtype == "bf16" else 4
        extra = {"design_bytes": design_bytes(wl.hidden, wl.c_in, s, wl.useful_cells, run.n_cells, run.unit_cells)}
        crit = max(int(h) + int(w) - 1 for h, w in zip(wl.heights, wl.widths))
    print(f"[bench] workload {cid} packed: {ms:.3f} ms/step (wall {wall_ms:.3f}), dominant kernel {dom} "
          f"{phase[dom]:.3f} ms", file=sys.stderr, flush=True)
    phases_out = phase_rates(phase, alg, dtype, f"workload {cid}")
    traffic = measured_traffic(dom, cid)
    roof = roofline(dom, phase[dom], *alg[dom], dtype, traffic)
    proj = projection_fractions(phase[proj_name], *alg[proj_name], dtype) if phase.get(proj_name) else None
    if proj is not None:
        proj["kernel"] = proj_name
    res = {
        "workload": name, "config": cid, "examples": wl.n, "dtype": dtype, "forward_only": forward_only,
        "value": useful / (ms * 1e-3), "unit": "cell-updates/s", "ms_per_step": round(ms, 4),
        "median_ms": round(float(np.median(per_step)), 4), "min_ms": round(float(np.min(per_step)), 4),
        "wall_ms_per_step": round(wall_ms, 4), "steps": steps, "useful_cell_dirs": useful,
        "canvas": [run.canvas_h, run.canvas_w], "critical_path_diagonals": crit,
        "roofline": roof, "projection": proj, "phases": phases_out,
        "layout_ms": round(run.layout_ms, 3), "scatter_ms": round(run.scatter_ms, 3),
        "value_with_layout": useful / ((ms + run.layout_ms + run.scatter_ms) * 1e-3),
        # device memory held at most by the packed run (inputs, weights, outputs,
        # gradients, workspace), the quantity the paper's Table IV reports per GPU
        "peak_memory_MB": round(peak_mb, 1),
    }
    res.update(extra)
    if stepwise and cid != 4:
        sw = run.time_stepwise_forward(max(3, steps // 2), warmup)
        res["wavefront_fwd_stepwise_graph_ms"] = round(sw, 4)
        print(f"[bench] forward wavefront, one launch per diagonal from a HIP graph: {sw:.3f} ms", file=sys.stderr,
              flush=True)
    del run
    if padded:
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        pr = RunCls(wl, "padded")
        pms, _, pphase, pper, _ = pr.time(max(3, steps // 2), warmup)
        ppeak = torch.cuda.max_memory_allocated() / 2**20
        res["padded"] = {"ms_per_step": round(pms, 4), "median_ms": round(float(np.median(pper)), 4),
                         "value": useful / (pms * 1e-3), "canvas_cells": pr.n_cells, "unit_cells": pr.unit_cells,
                         "speedup_packed_vs_padded": round(pms / ms, 3),
                         "padded_over_useful_cells": round(pr.unit_cells * 4 / useful, 3),
                         "layout_ms": round(pr.layout_ms + pr.scatter_ms, 3),
                         "peak_memory_MB": round(ppeak, 1),
                         "phases_ms": {k: round(v, 4) for k, v in pphase.items()}}
        print(f"[bench] workload {cid} padded: {pms:.3f} ms/step", file=sys.stderr, flush=True)
        del pr
    torch.cuda.empty_cache()
    return res


def measure_head(steps: int, warmup: int):
    """The shared output layer, row collapse and CTC loss on the word batch's
    packed canvas (80 classes, synthetic labels): head forward, CTC loss and
    gradient, head backward, each timed with events on the stream."""
    import torch

    from paper_1902_11208_amd import api
    from synth import configs

    wl = configs.workload(2)
    rects, ch, _ = api.pack_layout(wl.heights, wl.widths, wl.canvas_w)
    g = torch.Generator(device="cuda")
    g.manual_seed(2)
    y = torch.randn((ch, wl.canvas_w, 4 * wl.hidden), device="cuda", generator=g) * 0.3
    W, b = (torch.from_numpy(t).cuda() for t in wl.head_params())
    labels = [wl.label(k) for k in range(wl.n)]
    hd = api.Head(W, b, rects, (ch, wl.canvas_w), labels)
    for _ in range(warmup):
        hd.forward(y)
        hd.ctc()
        hd.backward()
    evs = [_events(torch, 4) for _ in range(steps)]
    torch.cuda.synchronize()
    for e in evs:
        e[0].record()
        hd.forward(y)
        e[1].record()
        hd.ctc()
        e[2].record()
        hd.backward()
        e[3].record()
    torch.cuda.synchronize()
    ms = {n: float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs]))
          for i, n in enumerate(("head_forward", "ctc", "head_backward"))}
    H, K = wl.hidden, W.shape[0]
    U, F = wl.useful_cells, int(np.sum(wl.widths))
    S = sum(2 * len(l) + 1 for l in labels)
    TS = int(sum(int(w) * (2 * len(l) + 1) for w, l in zip(wl.widths, labels)))
    # cost model: the forward reads the examples' cells once and writes the
    # logits; CTC reads the logits and writes their gradient (its forward and
    # backward variables, T x S doubles each way, stay in the caches when they
    # can); the backward writes the layer's upstream gradient over the examples
    alg = {"head_forward": (U * 4 * H * 4 + F * K * 4, U * 4 * H + 2.0 * F * K * H),
           "ctc": (2 * F * K * 4 + 2 * TS * 8, 30.0 * TS + 10.0 * F * K),
           "head_backward": (U * 4 * H * 4 + F * K * 4 + F * (H + 4) * 4, 2.0 * F * K * H + 2.0 * F * K * (H + 1))}
    dom = max(ms, key=lambda k: ms[k])
    by, fl = alg[dom]
    gbs = by / (ms[dom] * 1e-3) / 1e9
    out = {"workload": "word batch (256 x h16, H 16) output layer shared by the directions, row collapse, CTC loss "
                       f"with {K} classes and synthetic labels",
           "frames": F, "label_states": S, "ms_per_step": round(sum(ms.values()), 4),
           "phases": phase_rates(ms, alg, "f32", "head"),
           "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": None, "kernel": dom,
                        "ms": round(ms[dom], 4), "bytes_per_launch": int(by), "flops_per_launch": int(fl),
                        "note": "the CTC recursion walks the frames in order; its floor is the longest "
                                "example's frames times a step's latency, not bandwidth"
                        if dom == "ctc" else None}}
    print(f"[bench] output layer + CTC on the word batch: {out['ms_per_step']:.3f} ms "
          f"({', '.join(f'{k} {v:.3f}' for k, v in ms.items())})", file=sys.stderr, flush=True)
    return out


def measured_traffic(kernel: str, cid: int):
    """HBM bytes per launch of `kernel` on workload `cid` from the committed
    hardware-counter summary, or None when there is none or the kernel source
    changed since it was taken."""
    import glob
    import hashlib

    for path in glob.glob(os.path.join(ROOT, "profiles", "traffic_*.md")):
        fields = {}
        for line in open(path):
            if ":" in line and not line.startswith(("|", "#", " ")):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
        if fields.get("kernel") != kernel or fields.get("config") != str(cid):
            continue
        ok = True
        for k, v in fields.items():
            if k.startswith("source_sha256"):
                src = k[k.index("(") + 1:k.index(")")]
                ok &= hashlib.sha256(open(os.path.join(ROOT, src), "rb").read()).hexdigest() == v
        if ok:
            return int(fields["traffic_bytes_per_launch"])
    return None


# ---------------------------------------------------------------------------
# CPU baseline: the oracle on the host cores (before the GPU is touched)
# ---------------------------------------------------------------------------
def host_info():
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    aff = sorted(os.sched_getaffinity(0))
    return {"cpu_model": model, "nproc": os.cpu_count(), "affinity_cpus": len(aff)}


def _cpu_sample(cid: int, one_core: bool):
    """(label, run(workers) -> seconds, useful cell-updates) of a bounded
    sample of workload cid for the oracle."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle_run
    from synth import configs

    if cid == 4:
        wl = configs.stack_workload()
        ks = list(range(8 if one_core else wl.n))
        layers, convs = wl.params()
        imgs, dys = [wl.image(k) for k in ks], [wl.dy(k) for k in ks]
        useful = 4 * sum(int(wl.heights[k] // wl.block[0] ** (l + 1)) * int(wl.widths[k] // wl.block[1] ** (l + 1))
                         for k in ks for l in range(3))

        def run(workers):
            t0 = time.perf_counter()
            oracle_run.run_stack(imgs, layers, convs, dys, wl.block, workers=workers)
            return time.perf_counter() - t0

        return f"images {ks[0]}-{ks[-1]} of {wl.n}, all three layers and both convolutions", run, useful
    wl = configs.workload(cid)
    crop = None
    if cid == 1:
        ks = list(range(wl.n))
    elif cid == 2:
        ks = list(range(128 if one_core else wl.n))
    elif cid == 3:
        ks = list(range(8 if one_core else wl.n))
    else:  # bf16 stress: a 48 x 192 crop of each sampled example
        ks, crop = list(range(3 if one_core else 32)), 192
    xs = [wl.example(k) for k in ks]
    dys = None if wl.forward_only else [wl.dy(k) for k in ks]
    if crop:
        xs = [x[:, :crop] for x in xs]
        dys = [d[:, :crop] for d in dys]
    useful = 4 * sum(int(x.shape[0]) * int(x.shape[1]) for x in xs)
    params = wl.params()

    def run(workers):
        t0 = time.perf_counter()
        oracle_run.run_layer(xs, params, dys, backward=not wl.forward_only, workers=workers)
        return time.perf_counter() - t0

    what = f"examples {ks[0]}-{ks[-1]} of {wl.n}" if len(ks) > 1 else f"example {ks[0]} of {wl.n}"
    if crop:
        what += f", each cropped to its first {crop} columns ({wl.heights[0]} x {crop} cells)"
    return what + (", forward only" if wl.forward_only else ", forward+backward"), run, useful


def _one_core_child(cid, cpu, conn):
    os.sched_setaffinity(0, {cpu})
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle_run

    oracle_run.single_threaded_blas()
    label, run, useful = _cpu_sample(cid, True)
    conn.send((label, run(1), useful))
    conn.close()


def cpu_baseline(cid: int, host: dict):
    """The oracle as it stands (float64 NumPy, each example alone) on a bounded
    sample: a process pool with one worker per core of the affinity set (at
    most 16), then one forked worker pinned to a single core."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle_run

    workers = oracle_run.default_workers()
    label, run, useful = _cpu_sample(cid, False)
    dt = run(workers)
    ctx = mp.get_context("fork")
    a, b = ctx.Pipe(duplex=False)
    p = ctx.Process(target=_one_core_child, args=(cid, sorted(os.sched_getaffinity(0))[0], b))
    p.start()
    label1, dt1, useful1 = a.recv()
    p.join()
    out = {"value": useful / dt, "unit": "cell-updates/s", "cores": workers, "kind": "oracle",
           "sample": f"{label}; float64 NumPy, process pool of {workers} (one BLAS thread each), {dt:.1f} s wall",
           "one_core": {"value": useful1 / dt1, "unit": "cell-updates/s", "cores": 1,
                        "sample": f"{label1}; one forked worker pinned to one core, one BLAS thread, {dt1:.1f} s"}}
    out.update(host)
    print(f"[bench] cpu oracle, workload {cid}: {out['value']:.3e} cell-updates/s on {workers} cores, "
          f"{out['one_core']['value']:.3e} on one", file=sys.stderr, flush=True)
    return out


# ---------------------------------------------------------------------------
def main():
    args = _parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: --gpus {args.gpus} (WORLD_SIZE {world}) is not supported; the layer has "
              "no multi-GPU path (examples would be split across GPUs with an all-reduce of the weight "
              "gradients)", file=sys.stderr)
        sys.exit(2)
    head = args.config
    cids = [head] + ([] if args.no_nested else [c for c in [HEADLINE] + NESTED if c != head])
    host = host_info()
    cpu = {}
    if not args.no_cpu:  # before anything touches the GPU
        for cid in cids:
            cpu[cid] = cpu_baseline(cid, host)

    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    from paper_1902_11208_amd import _lib

    if not os.path.exists(_lib.LIB_PATH):
        from paper_1902_11208_amd import build

        build.build()
    res = {}
    for i, cid in enumerate(cids):
        steps = args.steps if i == 0 else min(args.steps, 5 if cid == 5 else 10)
        res[cid] = measure_gpu(cid, steps, args.warmup, not args.no_padded, stepwise=(i == 0))
        res[cid]["cpu_baseline"] = cpu.get(cid)

    h = res[head]
    out = {
        "metric": METRIC,
        "value": h["value"],
        "unit": "cell-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": h["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": h["dtype"],
        "data": "synthetic",
        "config": {"workload": h["workload"], "examples": h["examples"], "canvas": h["canvas"],
                   "useful_cell_dirs": h["useful_cell_dirs"], "forward_only": h["forward_only"]},
        "roofline": h["roofline"],
        "cpu_baseline": h["cpu_baseline"],
    }
    for k in ("padded", "projection", "phases", "design_bytes", "layers", "wavefront_fwd_stepwise_graph_ms",
              "critical_path_diagonals", "median_ms", "min_ms", "layout_ms", "scatter_ms", "value_with_layout",
              "wall_ms_per_step", "peak_memory_MB"):
        if k in h:
            out[k] = h[k]
    out["configs"] = {str(cid): res[cid] for cid in cids[1:]}
    if not args.no_nested:
        out["head_ctc"] = measure_head(min(args.steps, 10), args.warmup)
    out["paper_context"] = PAPER_CONTEXT
    out["host"] = host
    if args.copy_calibration:
        a = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
