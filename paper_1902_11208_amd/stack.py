"""Multi-layer MDLSTM stack on packed canvases (Section V-B).

Every layer keeps its examples packed: images are block-reshaped into the
first canvas, each MDLSTM layer runs on its canvas, and a grouped block
convolution with tanh maps its output onto the next layer's canvas, where
each example is bh times lower and bw times narrower and packed anew. All
arithmetic runs in the library's kernels; this module only sequences the
C-ABI calls and owns the buffers.
"""
from __future__ import annotations

import numpy as np
import torch

from . import api


class MDLSTMStack:
    """MDLSTM(H0) -> [block conv + tanh -> MDLSTM(H_l)] ... on packed canvases (fp32).

    layers: [(wx, u, b)] device tensors per MDLSTM layer; convs: [(w, b)] per
    block convolution (len(layers) - 1). heights/widths: image sizes, each a
    multiple of the total block reduction. canvas_w: canvas width per layer.
    kind "padded" lays every layer out last-minute padded instead (tiles of
    the batch maximum, mask = true extents) for comparison.
    """

    def __init__(self, layers, convs, heights, widths, canvas_w, block=(2, 4), in_channels: int = 1,
                 device="cuda", kind: str = "packed"):
        if len(convs) != len(layers) - 1 or len(canvas_w) != len(layers):
            raise ValueError("need one convolution between consecutive layers and one canvas width per layer")
        self.bh, self.bw = block
        self.in_channels = int(in_channels)
        hs = np.asarray(heights, np.int64).reshape(-1)
        ws = np.asarray(widths, np.int64).reshape(-1)
        self.n = int(hs.size)
        self.layers, self.convs = [], []
        self.rects, self.canvas = [], []
        for li, (wx, u, b) in enumerate(layers):
            f = (self.bh ** (li + 1), self.bw ** (li + 1))
            if np.any(hs % f[0]) or np.any(ws % f[1]):
                raise ValueError(f"image sizes must be multiples of {f[0]}x{f[1]}")
            if kind == "packed":
                rects, ch, mask = api.pack_layout(hs // f[0], ws // f[1], int(canvas_w[li]), device=device)
                units, cw = rects, int(canvas_w[li])
            else:
                units, rects, ch, cw, mask = api.pad_layout(hs // f[0], ws // f[1], device=device)
            self.rects.append(rects)
            self.canvas.append((ch, cw))
            self.layers.append(api.MDLSTMLayer(wx, u, b, ch, cw, units, mask))
        for li, (w, b) in enumerate(convs):
            self.convs.append(api.BlockConv(w, b, self.rects[li], self.canvas[li], self.rects[li + 1],
                                            self.canvas[li + 1], self.bh, self.bw))

    def pack_input(self, images, stream=None) -> torch.Tensor:
        ch, cw = self.canvas[0]
        imgs = [im if im.dim() == 3 else im[:, :, None] for im in images]
        return api.pack_blocks(imgs, self.rects[0], ch, cw, self.bh, self.bw, stream=stream)

    def forward(self, x0: torch.Tensor, stream=None) -> torch.Tensor:
        """x0: first packed canvas (pack_input). Returns the last layer's output canvas."""
        x = x0
        for li, layer in enumerate(self.layers):
            y = layer.forward(x, stream)
            if li < len(self.convs):
                x = self.convs[li].forward(y, stream)
        return y

    def backward(self, dy_last: torch.Tensor, stream=None) -> torch.Tensor:
        """dy_last: gradient of the last output canvas. Returns the gradient of x0;
        weight gradients are left in each layer (dwx, du, db) and conv (dw, db)."""
        g = dy_last
        for li in range(len(self.layers) - 1, -1, -1):
            dx, _, _, _ = self.layers[li].backward(g, stream)
            if li > 0:
                g, _, _ = self.convs[li - 1].backward(dx, stream)
            else:
                g = dx
        return g

    def useful_cells(self) -> int:
        """Example pixels summed over the layers' canvases."""
        return int(sum(int(np.sum(r[:, 2].astype(np.int64) * r[:, 3])) for r in self.rects))
