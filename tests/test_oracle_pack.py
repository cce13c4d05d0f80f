"""Pins for the oracle's example-packing layout (Section V-A, Algorithm 1)."""
import numpy as np
import pytest

from conftest import read_fixture
from oracle import pack
from synth import configs


def _fixture():
    rows = read_fixture("pack_w10.txt")
    cw, n = map(int, rows[0])
    hs = list(map(int, rows[1]))
    ws = list(map(int, rows[2]))
    ch, msum = map(int, rows[3])
    rects = np.array([list(map(int, r)) for r in rows[4:4 + n]], np.int32)
    return cw, hs, ws, ch, msum, rects


def test_hand_worked_layout():
    cw, hs, ws, ch, msum, rects = _fixture()
    got, got_h = pack.pack_layout(hs, ws, cw)
    assert got_h == ch
    np.testing.assert_array_equal(got, rects)
    assert int(pack.make_mask(got, got_h, cw).sum()) == msum


def check_invariants(hs, ws, cw, rects, ch):
    hs = np.asarray(hs)
    ws = np.asarray(ws)
    n = len(hs)
    assert rects.shape == (n, 4)
    np.testing.assert_array_equal(rects[:, 2], hs)
    np.testing.assert_array_equal(rects[:, 3], ws)
    occ = np.zeros((ch + 2, cw + 2), np.int32)  # one-pixel guard ring
    for k, (y0, x0, h, w) in enumerate(rects):
        assert 0 <= y0 and y0 + h <= ch and 0 <= x0 and x0 + w <= cw
        assert np.all(occ[y0 + 1:y0 + h + 1, x0 + 1:x0 + w + 1] == 0), "rectangles overlap"
        occ[y0 + 1:y0 + h + 1, x0 + 1:x0 + w + 1] = k + 1
    # no two examples 4-adjacent: a separator pixel always lies between them
    for dy, dx in ((0, 1), (1, 0)):
        a = occ[1:ch + 1, 1:cw + 1]
        b = occ[1 + dy:ch + 1 + dy, 1 + dx:cw + 1 + dx]
        assert not np.any((a > 0) & (b > 0) & (a != b))
    mask = pack.make_mask(rects, ch, cw)
    assert int(mask.sum()) == int(np.sum(hs.astype(np.int64) * ws))
    # rows: examples sharing y0 share the height; rows separated by exactly one pixel
    row_y0 = sorted(set(int(v) for v in rects[:, 0]))
    prev_end = None
    rows = []
    for y0 in row_y0:
        members = [k for k in range(n) if rects[k, 0] == y0]
        assert len(set(int(hs[k]) for k in members)) == 1
        h = int(hs[members[0]])
        if prev_end is not None:
            assert y0 == prev_end + 1
        prev_end = y0 + h
        members.sort(key=lambda k: rects[k, 1])
        rows.append((h, members))
    if n:
        assert ch == prev_end
    # heights ascending from row to row (buckets visited in ascending order)
    assert all(rows[i][0] <= rows[i + 1][0] for i in range(len(rows) - 1))
    # greedy: along a row widths never increase, the first example of a row is
    # the widest left in its bucket, and a row that closes inside its bucket
    # leaves no remaining example of that bucket that would have fitted
    for ri, (h, members) in enumerate(rows):
        w_row = [int(ws[k]) for k in members]
        assert w_row == sorted(w_row, reverse=True)
        x = 0
        for j, k in enumerate(members):
            assert rects[k, 1] == (x + 1 if j else 0)
            x = rects[k, 1] + ws[k]
        later = [k for (hh, mm) in rows[ri + 1:] if hh == h for k in mm]
        if later:
            assert max(int(ws[k]) for k in later) <= w_row[0]
            assert all(x + 1 + ws[k] > cw for k in later)


@pytest.mark.parametrize("seed", range(20))
def test_invariants_random(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 40))
    cw = int(rng.integers(8, 80))
    hs = rng.integers(1, 5, n)
    ws = rng.integers(1, cw + 1, n)
    rects, ch = pack.pack_layout(hs, ws, cw)
    check_invariants(hs, ws, cw, rects, ch)


@pytest.mark.parametrize("cid", [1, 2, 3, 5])
def test_invariants_configs(cid):
    wl = configs.workload(cid)
    rects, ch = pack.pack_layout(wl.heights, wl.widths, wl.canvas_w)
    check_invariants(wl.heights, wl.widths, wl.canvas_w, rects, ch)


def test_word_batch_padding_share():
    # Section VI: without packing about 75% of word-batch pixels are padding
    wl = configs.workload(2)
    assert 0.65 < configs.padded_fraction(wl.heights, wl.widths) < 0.85


def test_errors_and_empty():
    with pytest.raises(pack.PackError) as e:
        pack.pack_layout([2, 2], [5, 11], 10)
    assert e.value.code == "TOO_WIDE"
    with pytest.raises(pack.PackError) as e:
        pack.pack_layout([0], [3], 10)
    assert e.value.code == "INVALID_ARG"
    with pytest.raises(pack.PackError) as e:
        pack.pack_layout([2], [-1], 10)
    assert e.value.code == "INVALID_ARG"
    rects, ch = pack.pack_layout([], [], 10)
    assert rects.shape == (0, 4) and ch == 0


def test_exact_fit_and_single_column():
    # an example exactly as wide as the canvas fills a row alone
    rects, ch = pack.pack_layout([1, 1, 1], [10, 4, 5], 10)
    np.testing.assert_array_equal(rects, [[0, 0, 1, 10], [2, 6, 1, 4], [2, 0, 1, 5]])
    assert ch == 3
    rects, ch = pack.pack_layout([3, 1], [1, 1], 1)
    np.testing.assert_array_equal(rects, [[2, 0, 3, 1], [0, 0, 1, 1]])
    assert ch == 5


def test_scatter_gather_roundtrip():
    rng = np.random.default_rng(0)
    hs, ws = [2, 3, 2], [4, 5, 3]
    rects, ch = pack.pack_layout(hs, ws, 9)
    ex = [rng.standard_normal((h, w, 2)) for h, w in zip(hs, ws)]
    canvas = pack.scatter(ex, rects, ch, 9, 2)
    assert np.count_nonzero(np.abs(canvas).sum(axis=2)) == sum(h * w for h, w in zip(hs, ws))
    for a, b in zip(pack.gather(canvas, rects), ex):
        np.testing.assert_array_equal(a, b)


def test_pad_layout():
    tiles, place, ch, cw = pack.pad_layout([2, 3, 1], [4, 2, 5])
    assert (ch, cw) == (9, 5)
    np.testing.assert_array_equal(tiles, [[0, 0, 3, 5], [3, 0, 3, 5], [6, 0, 3, 5]])
    np.testing.assert_array_equal(place, [[0, 0, 2, 4], [3, 0, 3, 2], [6, 0, 1, 5]])
