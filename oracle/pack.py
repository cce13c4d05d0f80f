"""Example packing (Section V-A, Algorithm 1 in Appendix B) — oracle.

Test infrastructure only (see ``oracle/__init__.py``).

The paper's four steps: (1) bucket the examples by height, (2) inside each
bucket fill rows by repeatedly adding the widest example that still fits,
(3) tile the examples within rows and the rows on top of each other with one
separating pixel in between, (4) skew. The skew is index arithmetic only and
is never materialised here; canvases are kept unskewed.

Readings where the paper is silent or its pseudocode is inconsistent:

* buckets are visited in ascending height;
* "widest still fitting": candidates ordered by (width descending, original
  index ascending), the first that fits is taken;
* fit test: an empty row takes any example with w <= W; otherwise the example
  needs used + 1 + w <= W (a separator only sits between two examples);
* the row under construction is closed when nothing in the bucket fits, and is
  also flushed when the bucket runs empty (the printed pseudocode never emits
  the last row and would carry it into the next bucket, mixing heights, which
  the text forbids);
* x0 of the j-th example of a row is sum over earlier examples of (w + 1);
  y0 of row r is sum over earlier rows of (row height + 1); the canvas width
  is the given width, the canvas height is the sum of row heights plus one
  separator row between consecutive rows;
* mask = 1 exactly on example pixels; canvas values outside examples are 0;
* any example wider than the canvas is an error (the pseudocode would loop
  forever); non-positive sizes are errors; an empty list packs to height 0.
"""
from __future__ import annotations

import numpy as np


class PackError(ValueError):
    """Invalid packing request. ``code`` is 'TOO_WIDE' or 'INVALID_ARG'."""

    def __init__(self, code: str, msg: str):
        super().__init__(f"{code}: {msg}")
        self.code = code


def pack_layout(heights, widths, canvas_w: int):
    """Place examples on a canvas of width ``canvas_w``.

    Returns (rects, canvas_h): rects is int32 [n, 4] with rows (y0, x0, h, w),
    indexed by ORIGINAL example index.
    """
    hs = [int(v) for v in np.asarray(heights).reshape(-1)]
    ws = [int(v) for v in np.asarray(widths).reshape(-1)]
    if len(hs) != len(ws):
        raise PackError("INVALID_ARG", "heights and widths differ in length")
    if canvas_w <= 0:
        raise PackError("INVALID_ARG", "canvas width must be positive")
    for k, (h, w) in enumerate(zip(hs, ws)):
        if h <= 0 or w <= 0:
            raise PackError("INVALID_ARG", f"example {k} has size {h}x{w}")
        if w > canvas_w:
            raise PackError("TOO_WIDE", f"example {k} is {w} wide, canvas is {canvas_w}")
    n = len(hs)

    # Step 1: bucket by height (ascending).
    # Step 2: fill rows greedily with the widest example that still fits.
    rows = []  # list of (row_height, [original indices in placement order])
    for hb in sorted(set(hs)):
        bucket = sorted((k for k in range(n) if hs[k] == hb), key=lambda k: (-ws[k], k))
        current, used = [], 0
        while bucket:
            pick, need = None, 0
            for k in bucket:
                need = ws[k] if not current else used + 1 + ws[k]
                if need <= canvas_w:
                    pick = k
                    break
            if pick is not None:
                current.append(pick)
                used = need
                bucket.remove(pick)
            else:
                rows.append((hb, current))
                current, used = [], 0
        if current:
            rows.append((hb, current))

    # Step 3: tile within rows, then across rows, with one separating pixel.
    rects = np.zeros((n, 4), dtype=np.int32)
    y = 0
    for r, (hb, members) in enumerate(rows):
        if r > 0:
            y += 1
        x = 0
        for j, k in enumerate(members):
            if j > 0:
                x += 1
            rects[k] = (y, x, hb, ws[k])
            x += ws[k]
        y += hb
    return rects, y


def make_mask(rects, canvas_h: int, canvas_w: int) -> np.ndarray:
    """uint8 [canvas_h, canvas_w]: 1 on example pixels, 0 on separators and slack."""
    mask = np.zeros((canvas_h, canvas_w), dtype=np.uint8)
    for y0, x0, h, w in np.asarray(rects).reshape(-1, 4):
        mask[y0:y0 + h, x0:x0 + w] = 1
    return mask


def scatter(examples, rects, canvas_h: int, canvas_w: int, c: int, dtype=np.float64):
    """Copy each example [h, w, c] into its rectangle of a zero [H_c, W_c, c] canvas."""
    canvas = np.zeros((canvas_h, canvas_w, c), dtype=dtype)
    for ex, (y0, x0, h, w) in zip(examples, np.asarray(rects).reshape(-1, 4)):
        canvas[y0:y0 + h, x0:x0 + w] = ex
    return canvas


def gather(canvas, rects):
    """Inverse of ``scatter``: list of per-example views of the canvas (copies)."""
    return [np.array(canvas[y0:y0 + h, x0:x0 + w]) for y0, x0, h, w in np.asarray(rects).reshape(-1, 4)]


def pad_layout(heights, widths):
    """Last-minute batch padding (Section VI-B): every example is padded to the
    batch's maximum height and width.

    Tiles of h_max x w_max are stacked vertically with no separators; example k
    sits at the top-left of tile k. Returns (tiles, placements, canvas_h,
    canvas_w): tiles are the scheduling rectangles (state restarts at tile
    edges), placements the example rectangles (the mask).
    """
    hs = np.asarray(heights, np.int64).reshape(-1)
    ws = np.asarray(widths, np.int64).reshape(-1)
    n = hs.size
    if n == 0:
        z = np.zeros((0, 4), np.int32)
        return z, z.copy(), 0, 0
    hm, wm = int(hs.max()), int(ws.max())
    tiles = np.array([(k * hm, 0, hm, wm) for k in range(n)], dtype=np.int32).reshape(n, 4)
    place = np.array([(k * hm, 0, int(hs[k]), int(ws[k])) for k in range(n)], dtype=np.int32).reshape(n, 4)
    return tiles, place, n * hm, wm
