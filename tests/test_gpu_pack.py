"""GPU packing kernels (placement, mask, scatter, gather) are bit-exact with the oracle."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu(built_lib):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _cases():
    from synth import configs

    out = []
    for cid in (1, 2, 3, 5):
        wl = configs.workload(cid)
        out.append((f"config{cid}", wl.heights, wl.widths, wl.canvas_w))
    rng = np.random.default_rng(0)
    for i in range(6):
        n = int(rng.integers(1, 300))
        cw = int(rng.integers(8, 300))
        out.append((f"random{i}", rng.integers(1, 9, n), rng.integers(1, cw + 1, n), cw))
    out.append(("single", np.array([3]), np.array([7]), 7))
    out.append(("ties", np.array([2, 2, 2, 2, 2]), np.array([3, 3, 3, 3, 3]), 7))
    # the placement keeps a bit per sorted example, 64 per lane of one wave:
    # word boundaries and the largest packing call (4096 examples), with many
    # height buckets and with a single one
    rng = np.random.default_rng(3)
    out.append(("n64", rng.integers(1, 4, 64), rng.integers(1, 51, 64), 50))
    out.append(("n65", rng.integers(1, 4, 65), rng.integers(1, 51, 65), 50))
    out.append(("max_n_buckets", rng.integers(1, 41, 4096), rng.integers(1, 65, 4096), 512))
    out.append(("max_n_one_bucket", np.full(4096, 5), rng.integers(1, 65, 4096), 1024))
    return out


CASES = _cases()


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_layout_and_mask_bitexact(case):
    from oracle import pack
    from paper_1902_11208_amd import api

    name, hs, ws, cw = case
    print(f"pack case {name}: n={len(hs)} W={cw}", flush=True)
    sys.stdout.flush()
    rects, ch, mask = api.pack_layout(hs, ws, cw)
    ref, ref_h = pack.pack_layout(hs, ws, cw)
    assert ch == ref_h
    np.testing.assert_array_equal(rects, ref)
    np.testing.assert_array_equal(mask.cpu().numpy(), pack.make_mask(ref, ref_h, cw))


def test_pad_layout_and_mask():
    from oracle import pack
    from paper_1902_11208_amd import api

    hs, ws = [3, 5, 2], [7, 4, 9]
    tiles, place, ch, cw, mask = api.pad_layout(hs, ws)
    rt, rp, rh, rw = pack.pad_layout(hs, ws)
    assert (ch, cw) == (rh, rw)
    np.testing.assert_array_equal(tiles, rt)
    np.testing.assert_array_equal(place, rp)
    np.testing.assert_array_equal(mask.cpu().numpy(), pack.make_mask(rp, rh, rw))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_scatter_gather_bitexact(dtype):
    import gpu_run
    from oracle import pack
    from paper_1902_11208_amd import api

    rng = np.random.default_rng(1)
    hs, ws, C = [3, 5, 2, 4], [7, 4, 9, 1], 8
    rects, ch, _ = api.pack_layout(hs, ws, 12)
    ex = [rng.standard_normal((h, w, C)).astype(np.float32) for h, w in zip(hs, ws)]
    dev = [gpu_run.to_dev(e, dtype) for e in ex]
    canvas = api.pack_data(dev, rects, ch, 12)
    ref = pack.scatter([d.float().cpu().numpy() for d in dev], rects, ch, 12, C)
    np.testing.assert_array_equal(canvas.float().cpu().numpy(), ref)
    back = api.unpack_data(canvas, rects)
    for a, b in zip(back, dev):
        assert torch.equal(a, b)
