"""Workload definitions and seeded draws.

The paper measures on IAM word-strips and line-strips (Section VI, Table IV).
Those images are not available here, so every workload is synthetic: example
heights and widths follow the shape of word-like and line-like batches, pixel
values and weights come from fixed distributions, and every tensor is drawn
from its own seeded stream so any single example can be regenerated without
drawing the rest.

Stream keys: ``SeedSequence([config_id, tag, index])`` with tag
0 = example sizes, 1 = example input, 2 = layer parameters, 3 = upstream
gradient. Values are drawn in float64, then rounded to float32 (and further to
bfloat16, round-to-nearest-even, for the bf16 workload).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

TAG_SIZES, TAG_INPUT, TAG_PARAMS, TAG_DY, TAG_LABELS = 0, 1, 2, 3, 4

# classes of the output layer: the CTC blank (class 0) and 79 symbols, close to
# the character set of the handwriting the paper trains on
HEAD_CLASSES = 80


def _rng(cid: int, tag: int, index: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([cid, tag, index]))


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returned as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + lsb) >> 16) << 16
    out = rounded.astype(np.uint32).view(np.float32)
    # NaN stays NaN (not produced by these draws, kept for completeness)
    return np.where(np.isnan(a), a, out)


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    a32 = np.asarray(a, dtype=np.float32)
    return round_to_bf16(a32) if dtype == "bf16" else a32


@dataclass
class Workload:
    """One MDLSTM layer over a batch of variable-size examples."""

    cid: int
    name: str
    dtype: str  # storage dtype: "f32" or "bf16" (accumulation is always fp32)
    heights: np.ndarray  # int32 [n]
    widths: np.ndarray  # int32 [n]
    canvas_w: int
    c_in: int
    hidden: int
    forward_only: bool
    forget_bias: float = -1.0  # centre of the two forget-gate biases (see params)

    @property
    def n(self) -> int:
        return int(self.heights.shape[0])

    @property
    def useful_cells(self) -> int:
        return int(np.sum(self.heights.astype(np.int64) * self.widths.astype(np.int64)))

    def example(self, k: int) -> np.ndarray:
        """Input of example k, [h, w, c_in] float32 (bf16-representable for bf16)."""
        h, w = int(self.heights[k]), int(self.widths[k])
        x = _rng(self.cid, TAG_INPUT, k).standard_normal((h, w, self.c_in))
        return _store(x, self.dtype)

    def examples(self, ks=None) -> list:
        ks = range(self.n) if ks is None else ks
        return [self.example(k) for k in ks]

    def params(self):
        """Per-direction weights: Wx [4][5H][c_in], U [4][5H][2H], b [4][5H] (float32).

        Gate order along the 5H axis: input gate, left forget gate, top forget
        gate, output gate, cell candidate. U's first H columns read the left
        predecessor's hidden state, the last H the top predecessor's.

        Every weight and bias is U(-0.1, 0.1); the biases of the two forget
        gates are then shifted by `forget_bias`. With a shift of 0 the two
        forget gates sum to about 1 and the plain cell's state grows without
        bound along long scans (|c| ~ 1e5 on 600-wide lines, ~1e16 on
        1200-wide ones); a shift of -1 keeps f_L + f_T near 0.54 and the state
        bounded.
        """
        H, C = self.hidden, self.c_in
        rng = _rng(self.cid, TAG_PARAMS, 0)
        wx, u, b = [], [], []
        for _d in range(4):
            wx.append(rng.uniform(-0.1, 0.1, (5 * H, C)))
            u.append(rng.uniform(-0.1, 0.1, (5 * H, 2 * H)))
            bd = rng.uniform(-0.1, 0.1, (5 * H,))
            bd[H:3 * H] += self.forget_bias
            b.append(bd)
        return (_store(np.stack(wx), self.dtype), _store(np.stack(u), self.dtype),
                _store(np.stack(b), self.dtype))

    def memory_params(self) -> np.ndarray:
        """Memory-state matrices V [4][3H][2H] (rows i, f_L, f_T; columns c_L,
        c_T), U(-0.1, 0.1), in the storage dtype."""
        rng = _rng(self.cid, TAG_PARAMS, 2)
        return _store(rng.uniform(-0.1, 0.1, (4, 3 * self.hidden, 2 * self.hidden)), self.dtype)

    def label(self, k: int, classes: int = HEAD_CLASSES) -> np.ndarray:
        """Target sequence of example k for the CTC loss: length U{1..max(1, w // 4)}
        (short enough for every frame path to exist, repeats included), classes
        U{1..classes-1} (0 is the blank). int32."""
        w = int(self.widths[k])
        rng = _rng(self.cid, TAG_LABELS, k)
        n = int(rng.integers(1, max(1, w // 4), endpoint=True))
        return rng.integers(1, classes, n, endpoint=False).astype(np.int32)

    def head_params(self, classes: int = HEAD_CLASSES):
        """Output layer shared by the directions: W [classes][H], b [classes], U(-0.1, 0.1), float32."""
        rng = _rng(self.cid, TAG_PARAMS, 1)
        W = rng.uniform(-0.1, 0.1, (classes, self.hidden))
        b = rng.uniform(-0.1, 0.1, (classes,))
        return _store(W, "f32"), _store(b, "f32")

    def dy(self, k: int) -> np.ndarray:
        """Upstream gradient of example k, [h, w, 4H] float32, N(0,1)."""
        h, w = int(self.heights[k]), int(self.widths[k])
        g = _rng(self.cid, TAG_DY, k).standard_normal((h, w, 4 * self.hidden))
        return _store(g, self.dtype)


def _sizes_config1():
    rng = _rng(1, TAG_SIZES)
    n = 4
    hs = rng.integers(8, 16, size=n, endpoint=True)
    ws = rng.integers(8, 32, size=n, endpoint=True)
    return hs, ws


def _sizes_config2():
    rng = _rng(2, TAG_SIZES)
    n = 256
    hs = np.full(n, 16)
    ws = np.clip(np.rint(rng.lognormal(np.log(40.0), 0.6, size=n)), 8, 200)
    return hs, ws


def _sizes_config3():
    rng = _rng(3, TAG_SIZES)
    n = 64
    hs = np.full(n, 32)
    ws = rng.integers(200, 600, size=n, endpoint=True)
    return hs, ws


def _sizes_config5():
    rng = _rng(5, TAG_SIZES)
    n = 128
    hs = np.full(n, 48)
    ws = rng.integers(300, 1200, size=n, endpoint=True)
    return hs, ws


_LAYER_CONFIGS = {
    # cid: (name, dtype, sizes, canvas_w, c_in, hidden, forward_only)
    1: ("tiny: 4 examples, C_in 8, H 4, forward only", "f32", _sizes_config1, 64, 8, 4, True),
    2: ("words: 256 x h16 lognormal widths, C_in 16, H 16", "f32", _sizes_config2, 1024, 16, 16, False),
    3: ("lines: 64 x h32 widths 200-600, C_in 32, H 32", "f32", _sizes_config3, 2048, 32, 32, False),
    5: ("bf16 stress: 128 x h48 widths 300-1200, C_in 64, H 128", "bf16", _sizes_config5, 4096, 64, 128, False),
}


def workload(cid: int) -> Workload:
    """Single-layer workload `cid` in {1, 2, 3, 5}."""
    if cid not in _LAYER_CONFIGS:
        raise ValueError(f"no single-layer workload {cid}; the three-layer stack is stack_workload()")
    name, dtype, sizes, cw, c_in, hidden, fwd_only = _LAYER_CONFIGS[cid]
    hs, ws = sizes()
    # the tiny workload keeps all parameters U(-0.1, 0.1) as stated for it;
    # the others centre the forget-gate biases at -1
    return Workload(cid=cid, name=name, dtype=dtype, heights=np.asarray(hs, np.int32),
                    widths=np.asarray(ws, np.int32), canvas_w=cw, c_in=c_in, hidden=hidden,
                    forward_only=fwd_only, forget_bias=0.0 if cid == 1 else -1.0)


def custom_workload(cid: int, heights, widths, canvas_w: int, c_in: int, hidden: int,
                    dtype: str = "f32", forget_bias: float = -1.0) -> Workload:
    """A workload with explicit sizes (used for small test cases); draws keyed by `cid`."""
    return Workload(cid=cid, name=f"custom {cid}", dtype=dtype,
                    heights=np.asarray(heights, np.int32), widths=np.asarray(widths, np.int32),
                    canvas_w=int(canvas_w), c_in=int(c_in), hidden=int(hidden), forward_only=False,
                    forget_bias=float(forget_bias))


@dataclass
class StackWorkload:
    """Three MDLSTM layers with block-strided convolutions between them.

    A grey-scale line image (1 channel, pixels U(0,1)) is cut into 2x4 blocks
    (height x width) to give 8 channels; then MDLSTM(H=16), a 2x4 block
    convolution to 32 channels with tanh (4 groups, one per direction), MDLSTM(H=32),
    a 2x4 block convolution to 64 channels with tanh, MDLSTM(H=64).
    """

    cid: int
    heights: np.ndarray  # image heights (64)
    widths: np.ndarray  # image widths (multiples of 64)
    hidden: tuple = (16, 32, 64)
    conv_out: tuple = (32, 64)
    block: tuple = (2, 4)
    canvas_w: tuple = (2048, 512, 128)
    mdlstm_c_in: tuple = field(default=(8, 32, 64))

    @property
    def n(self) -> int:
        return int(self.heights.shape[0])

    def image(self, k: int) -> np.ndarray:
        h, w = int(self.heights[k]), int(self.widths[k])
        return _store(_rng(self.cid, TAG_INPUT, k).uniform(0.0, 1.0, (h, w)), "f32")

    def params(self):
        """[(Wx, U, b) for each MDLSTM layer], [(W, b) for each block conv].

        Block conv weights: W [4 groups][out/4][bh*bw*H_prev] reading direction
        d's H_prev channels of a bh x bw block, input index (dy*bw + dx)*H_prev + j.
        """
        rng = _rng(self.cid, TAG_PARAMS, 0)
        layers, convs = [], []
        for li, (c_in, H) in enumerate(zip(self.mdlstm_c_in, self.hidden)):
            wx, u, b = [], [], []
            for _d in range(4):
                wx.append(rng.uniform(-0.1, 0.1, (5 * H, c_in)))
                u.append(rng.uniform(-0.1, 0.1, (5 * H, 2 * H)))
                bd = rng.uniform(-0.1, 0.1, (5 * H,))
                bd[H:3 * H] -= 1.0  # forget-gate biases centred at -1, as for the single layers
                b.append(bd)
            layers.append((_store(np.stack(wx), "f32"), _store(np.stack(u), "f32"),
                           _store(np.stack(b), "f32")))
            if li < 2:
                bh, bw = self.block
                og = self.conv_out[li] // 4
                W = rng.uniform(-0.1, 0.1, (4, og, bh * bw * H))
                bb = rng.uniform(-0.1, 0.1, (4, og))
                convs.append((_store(W, "f32"), _store(bb, "f32")))
        return layers, convs

    def out_shape(self, k: int):
        h, w = int(self.heights[k]), int(self.widths[k])
        bh, bw = self.block
        return h // bh ** 3, w // bw ** 3, 4 * self.hidden[2]

    def dy(self, k: int) -> np.ndarray:
        h3, w3, c3 = self.out_shape(k)
        return _store(_rng(self.cid, TAG_DY, k).standard_normal((h3, w3, c3)), "f32")


def stack_workload() -> StackWorkload:
    rng = _rng(4, TAG_SIZES)
    n = 32
    hs = np.full(n, 64)
    ws = rng.integers(400, 1600, size=n, endpoint=True)
    ws = ((ws + 63) // 64) * 64  # every stage divides: 64 = 4*4*4
    return StackWorkload(cid=4, heights=np.asarray(hs, np.int32), widths=np.asarray(ws, np.int32))


def padded_fraction(heights, widths) -> float:
    """Share of cells that are padding when every example is padded to the batch maximum."""
    hs = np.asarray(heights, np.int64)
    ws = np.asarray(widths, np.int64)
    if hs.size == 0:
        return 0.0
    return 1.0 - float(np.sum(hs * ws)) / float(hs.size * hs.max() * ws.max())
