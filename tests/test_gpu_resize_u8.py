"""GPU parity of the uint8 cache writer (vp_resize_batch).

The fixed-point resampler is integer arithmetic from the 22-bit weights on,
so the device bytes must equal the oracle's exactly (the oracle itself is
pinned byte for byte to Pillow's bicubic resize): small cases in full, and
sampled frames of the full-size 64 x 256-frame workload and of the ragged
image/video batch.  Bytes beyond the batch must stay untouched.
"""
import sys

import numpy as np
import pytest

import oracle
import paper_2604_16893_amd as vp
import workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def log(msg):
    print(f"[gpu-resize-u8] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def run(items, sentinel=8, patch=16):
    """items: list of (device frames, indices, h, w).  Returns the output
    buffer (without the sentinel bytes) and frame_off."""
    vitems = [vp.Item(f, idx, h, w, patch) for f, idx, h, w in items]
    off, ws = vp.vp_resize_layout(vitems)
    total = int(off[-1])
    out = torch.full((total + sentinel,), 0xA5, dtype=torch.uint8, device=DEV)
    work = torch.empty(max(ws, 1), dtype=torch.uint8, device=DEV)
    off2 = vp.vp_resize_batch(vitems, out, work)
    torch.cuda.synchronize()
    assert off2.tolist() == off.tolist()
    assert (out[total:] == 0xA5).all(), "bytes beyond the batch were written"
    return out[:total], off


def frames_of(out, off, k, n, h, w):
    return out[int(off[k]):int(off[k + 1])].view(n, h, w, 3)


def _video(seed, n, H, W, gen="uniform"):
    it = workloads.Item("video", n, H, W, gen, seed, {"mode": "uniform", "n": n})
    return it, workloads.frames_torch(it, DEV)


CASES = [
    # name, [(n_src, H, W, indices, h, w)]
    ("downscale_2x", [(3, 64, 96, [2, 0], 32, 48 + 16)]),
    ("upscale_1_6x", [(2, 40, 50, [1, 0, 1], 64, 96)]),
    ("upscale_2x_eight_slots", [(2, 48, 80, [1, 0], 96, 160)]),
    ("upscale_2_5x_tiles", [(1, 64, 64, [0], 160, 160)]),
    ("identity", [(2, 64, 96, [1], 64, 96)]),
    ("mixed_axes", [(2, 100, 60, [0, 1], 64, 96)]),
    ("odd_width_854", [(2, 60, 854, [1, 0], 32, 640)]),
    ("tall_strong_downscale", [(2, 2400, 100, [1, 0], 64, 32)]),
    ("wide_strong_downscale", [(1, 300, 3000, [0], 32, 96)]),
    ("long_window_4k_width", [(2, 540, 3840, [1, 0], 96, 672)]),
    # x downscale of 3.9x: 16-column blocks read more than 64 pixels, so the
    # byte dot-product kernel takes it instead of the matrix-core one
    ("dot4_kernel_3_9x", [(2, 100, 1000, [0, 1], 64, 256)]),
    # matrix-core horizontal pass (windows of 10+ taps) with a vertical
    # upscale that keeps seven rows open
    ("mfma_seven_slots", [(2, 40, 240, [1, 0], 64, 96)]),
    # matrix-core form on rows and frames that start off 4-byte boundaries
    # (3 W = 783 bytes per row, 58,725 bytes per frame)
    ("mfma_unaligned_rows", [(3, 75, 261, [2, 0, 1], 32, 96)]),
    ("single_pixel", [(1, 1, 1, [0], 32, 32)]),
    ("ragged_batch", [(4, 75, 101, [3, 1, 2], 64, 96), (1, 333, 257, [0], 320, 256),
                      (5, 120, 200, [4, 0], 96, 160)]),
]


@pytest.mark.parametrize("name,specs", CASES, ids=[c[0] for c in CASES])
def test_resize_u8_small_cases_exact(name, specs):
    items, hosts = [], []
    for k, (n, H, W, idx, h, w) in enumerate(specs):
        it, fd = _video(400 + k, n, H, W)
        items.append((fd, np.asarray(idx, np.int32), h, w))
        hosts.append(workloads.frames_np(it))
    log(f"case {name}: {[(s[0], s[1], s[2], s[4], s[5]) for s in specs]}")
    out, off = run(items)
    for k, (fd, idx, h, w) in enumerate(items):
        got = frames_of(out, off, k, len(idx), h, w).cpu().numpy()
        ref = oracle.resize_u8_item(hosts[k], idx, h, w)
        diff = int((got != ref).sum())
        log(f"{name} item {k}: {diff} differing bytes of {ref.size}")
        assert diff == 0


def _sampled_workload_check(wl, n_check, seed):
    items = []
    for it in wl.items:
        if it.dims is not None:
            h, w = it.dims
        else:
            h, w = vp.vp_smart_resize_dims(it.H, it.W, 32, it.min_pixels, it.max_pixels)
        idx = vp.vp_sample_indices(it.n_src, vp.VP_SAMPLE_UNIFORM, it.sample["n"])
        items.append((workloads.frames_torch(it, DEV, chunk=32), idx, h, w))
    out, off = run(items, sentinel=4)
    rng = np.random.default_rng(seed)
    for _ in range(n_check):
        k = int(rng.integers(0, len(items)))
        fd, idx, h, w = items[k]
        m = int(rng.integers(0, len(idx)))
        got = frames_of(out, off, k, len(idx), h, w)[m].cpu().numpy()
        ref = oracle.resize_u8(workloads.frames_np(wl.items[k], [idx[m]])[0], h, w)
        diff = int((got != ref).sum())
        log(f"{wl.name[:3]} item {k} frame {m}: {diff} differing bytes")
        assert diff == 0
    del items, out


def test_resize_u8_rollout_workload_full_size():
    _sampled_workload_check(workloads.config(4), 6, 51)


def test_resize_u8_ragged_workload_full_size():
    _sampled_workload_check(workloads.config(3), 10, 52)


def test_resize_u8_patch14_widths():
    """Sizes on the patch-14 grid (multiples of 28): column bands of 64 that
    end in a 60-column band (252) or a 48-column one (112), so the stage
    leaves 45 and 36 dwords per band row."""
    specs = [(1, 333, 257, [0], 308, 252), (3, 70, 90, [2, 0, 1], 56, 112), (2, 720, 1280, [1, 0], 252, 448)]
    items, hosts = [], []
    for k, (n, H, W, idx, h, w) in enumerate(specs):
        it, fd = _video(470 + k, n, H, W)
        items.append((fd, np.asarray(idx, np.int32), h, w))
        hosts.append(workloads.frames_np(it))
    log(f"case patch14_widths: {[(s[0], s[1], s[2], s[4], s[5]) for s in specs]}")
    out, off = run(items, patch=14)
    for k, (fd, idx, h, w) in enumerate(items):
        got = frames_of(out, off, k, len(idx), h, w).cpu().numpy()
        ref = oracle.resize_u8_item(hosts[k], idx, h, w, patch=14)
        diff = int((got != ref).sum())
        log(f"patch14_widths item {k}: {diff} differing bytes of {ref.size}")
        assert diff == 0

