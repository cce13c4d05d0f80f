"""The allocation-free placement (mdlstm_pack_layout_noalloc, static device
scratch) against mdlstm_pack_layout (caller workspace): identical rectangles,
canvas height and mask bytes, on two calls in a row, the second one smaller,
so the second reuses the scratch the first left behind."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _sizes(seed, n, h_lo, h_hi, w_lo, w_hi):
    rng = np.random.default_rng(seed)
    return rng.integers(h_lo, h_hi + 1, n).tolist(), rng.integers(w_lo, w_hi + 1, n).tolist()


@pytest.fixture(scope="module", autouse=True)
def _need_gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_pack_layout_noalloc_matches_pack_layout():
    from paper_1902_11208_amd import api
    from synth import configs

    wl = configs.workload(2)
    cases = [("word batch, 256 examples", wl.heights.tolist(), wl.widths.tolist(), wl.canvas_w),
             ("37 random examples", *_sizes(71, 37, 1, 40, 1, 150), 200)]
    for label, hs, ws, cw in cases:
        print(f"case: allocation-free placement, {label}, canvas width {cw}", flush=True)
        ref_rects, ref_h, ref_mask = api.pack_layout(hs, ws, cw)
        max_h = int(np.sum(np.asarray(hs) + 1))
        buf = torch.full((max_h * cw,), 0xAB, dtype=torch.uint8, device="cuda")
        rects, ch = api.pack_layout_noalloc(hs, ws, cw, mask=buf)
        torch.cuda.synchronize()
        assert ch == ref_h
        assert np.array_equal(rects, ref_rects)
        assert torch.equal(buf[:ch * cw].view(ch, cw), ref_mask)
        assert bool((buf[ch * cw:] == 0xAB).all()), "wrote past the mask"
        # placement only (no mask)
        rects2, ch2 = api.pack_layout_noalloc(hs, ws, cw)
        assert ch2 == ref_h and np.array_equal(rects2, ref_rects)
