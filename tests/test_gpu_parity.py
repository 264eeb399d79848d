"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Every case runs the native library (vp_smart_resize_dims, vp_sample_indices,
vp_batch_layout, vp_preprocess_batch) on seeded synthetic frames resident on
the GPU and compares with the oracle on the same bytes: sizes, indices,
grid_thw and cu_seqlens bit-exact; pixel values within 2e-5 (float32) or one
bfloat16 ulp / 2e-5 (bfloat16).  Small cases are compared element by element
in full; the five workloads run at their full sizes, every row of the first
four checked against the oracle and, of the 64-video batch, eight whole
videos plus 100,352 rows sampled over all 64 (the oracle runs in a thread
pool); a NaN sentinel proves that every output row was written and none
beyond.
"""
import concurrent.futures as cf
import copy
import os
import sys

import numpy as np
import pytest

import oracle
from oracle import compare
import paper_2604_16893_amd as vp
import workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def log(msg):
    print(f"[gpu-parity] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# --------------------------------------------------------------------------
# helpers
# --------------------------------------------------------------------------

def plan_item(it: workloads.Item):
    """Target size and indices from the library, asserted bit-exact with the oracle."""
    if it.dims is not None:
        h, w = it.dims
    else:
        F = 2 * it.patch
        h, w = vp.vp_smart_resize_dims(it.H, it.W, F, it.min_pixels, it.max_pixels)
        assert (h, w) == oracle.smart_resize(it.H, it.W, F, it.min_pixels, it.max_pixels)
    s = it.sample
    if s["mode"] == "uniform":
        idx = vp.vp_sample_indices(it.n_src, vp.VP_SAMPLE_UNIFORM, s["n"])
        assert idx.tolist() == oracle.sample_uniform(it.n_src, s["n"]).tolist()
    else:
        idx = vp.vp_sample_indices(it.n_src, vp.VP_SAMPLE_FPS, 0, s["video_fps"], s["fps"],
                                   s["min_frames"], s["max_frames"])
        assert idx.tolist() == oracle.sample_fps(it.n_src, s["video_fps"], s["fps"],
                                                 s["min_frames"], s["max_frames"]).tolist()
    return h, w, idx


def run_gpu(items, mean, std, dtype, extra_rows=8, stream=None, patch=16):
    """items: list of (device frames, indices, h, w).  Output is prefilled
    with NaN and has `extra_rows` spare rows that must stay NaN."""
    vitems = [vp.Item(f, idx, h, w, patch) for f, idx, h, w in items]
    grid, cu, rows, ws = vp.vp_batch_layout(vitems)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = torch.full((rows + extra_rows, vp.row_width(patch)), float("nan"), dtype=tdt, device=DEV)
    work = torch.empty(ws, dtype=torch.uint8, device=DEV)
    g2, cu2 = vp.vp_preprocess_batch(vitems, mean, std,
                                     vp.VP_OUT_BF16 if dtype == "bf16" else vp.VP_OUT_F32,
                                     out, work, stream)
    assert g2.tolist() == grid.tolist() and cu2.tolist() == cu.tolist()
    torch.cuda.synchronize()
    og, ocu = oracle.layout([len(i[1]) for i in items], [i[2] for i in items],
                            [i[3] for i in items], patch=patch)
    assert grid.tolist() == og.tolist() and cu.tolist() == ocu.tolist()
    if extra_rows:
        assert torch.isnan(out[rows:].float()).all(), "rows beyond the batch were written"
    return out[:rows], grid, cu


def host_rows(out, lo, hi, dtype):
    t = out[lo:hi]
    if dtype == "bf16":
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def assert_close(gpu, ref, dtype, what):
    res = compare.check_bf16(gpu, ref) if dtype == "bf16" else compare.check_f32(gpu, ref)
    log(f"{what}: {res}")
    assert res["ok"], f"{what}: {res}"


def all_written(out):
    return not torch.isnan(out.float() if out.dtype == torch.bfloat16 else out).any().item()


# --------------------------------------------------------------------------
# generators: device and host copies agree
# --------------------------------------------------------------------------

@pytest.mark.parametrize("gen", ["uniform", "gradnoise", "rects"])
def test_device_generator_matches_host(gen):
    it = workloads.Item("video", 6, 97, 131, gen, 77, {"mode": "uniform", "n": 2},
                        rects=workloads._rects(5, 97, 131) if gen == "rects" else None)
    dev = workloads.frames_torch(it, DEV, chunk=4).cpu().numpy()
    assert np.array_equal(dev, workloads.frames_np(it))


# --------------------------------------------------------------------------
# small cases, compared in full
# --------------------------------------------------------------------------

def _rand_video(seed, n, H, W):
    return workloads.Item("video", n, H, W, "uniform", seed, {"mode": "uniform", "n": n})


SMALL = [
    # (name, [(n_src, H, W, indices, h, w)], dtype)
    ("identity_f32", [(2, 64, 96, [0, 1], 64, 96)], "f32"),
    ("identity_bf16", [(3, 64, 64, [2, 0], 64, 64)], "bf16"),
    ("upscale", [(2, 40, 50, [1, 0], 64, 96)], "f32"),
    ("single_pixel_source", [(1, 1, 1, [0], 32, 32)], "f32"),
    ("odd_stride_854", [(3, 60, 854, [0, 2], 32, 640)], "f32"),
    ("odd_count_and_image", [(5, 70, 90, [4, 1, 3], 64, 96), (1, 250, 333, [0], 256, 320)], "bf16"),
    ("repeated_unsorted", [(4, 50, 70, [3, 3, 0, 3, 1, 1], 32, 64)], "f32"),
    ("strong_downscale_subtiles", [(2, 300, 3000, [0, 1], 32, 96)], "f32"),
    ("tall_downscale", [(2, 2400, 100, [1, 0], 64, 32)], "bf16"),
    ("ragged_mixed", [(9, 120, 200, [0, 3, 8, 5], 96, 160), (1, 333, 257, [0], 320, 256),
                      (7, 45, 80, [6], 64, 64), (3, 480, 854, [0, 1, 2], 128, 224)], "bf16"),
    # streaming-kernel shapes: five accumulator slots with three pixels per
    # lane; a last column band of 32 after two of 64; odd frame sizes, so
    # that every other frame starts off a 4-byte boundary; a frame narrower
    # than one wave's pixels (lanes past the row end)
    ("slots5_px3", [(3, 224, 700, [2, 0], 160, 256)], "f32"),
    ("partial_band", [(2, 300, 450, [1, 0], 128, 160)], "bf16"),
    ("unaligned_frames", [(4, 75, 101, [1, 2, 3], 64, 96)], "f32"),
    ("narrow_frame", [(2, 100, 40, [0, 1], 64, 32)], "f32"),
    # vertical upscales on the streaming kernel (several output rows close
    # on one source row; 2x keeps eight rows open); a stronger one on the
    # general kernel, with an odd count whose padded pair is one frame twice
    ("upscale_stream", [(2, 60, 70, [1, 0], 64, 96)], "f32"),
    ("upscale_2x_eight_slots", [(2, 48, 80, [1, 0], 96, 160), (1, 120, 160, [0], 224, 288)], "bf16"),
    ("upscale_general_odd", [(3, 24, 40, [2, 0, 1], 64, 96)], "bf16"),
    # long x windows (downscales of 4x to 7x): 28 taps with two pixels per
    # lane in 16-column bands, 20 taps with three in 32-column bands, and a
    # 4K-wide frame (24 taps)
    ("long_window_28", [(2, 90, 1600, [1, 0], 32, 256)], "f32"),
    ("long_window_20_px3", [(3, 200, 1800, [2, 0], 64, 384)], "bf16"),
    ("long_window_4k_width", [(2, 540, 3840, [0, 1], 96, 672)], "bf16"),
    # tap counts that are not a multiple of 4 (the x pass's last group
    # holds 1 to 3 taps): 9 taps with two pixels per lane, 10 with three,
    # 7 in bf16
    ("taps9_px2", [(2, 180, 640, [1, 0], 96, 288)], "f32"),
    ("taps10_px3", [(3, 90, 300, [2, 0], 32, 128)], "bf16"),
    ("taps7_bf16", [(2, 120, 854, [1, 0], 64, 512)], "bf16"),
    # the x-first kernel (vertical scales up to 1.6): 12, 10 and 8 taps,
    # a last band of 32 columns, odd frame sizes (windows at every byte
    # alignment), a scale just under the limit; one just over it and a
    # near-1 vertical scale whose x window is too long for x-first stay on
    # the y-first kernel
    ("xfirst_taps12_ragged_band", [(2, 100, 691, [1, 0], 96, 288)], "f32"),
    ("xfirst_taps10_bf16", [(3, 90, 512, [2, 0, 1], 96, 256)], "bf16"),
    ("xfirst_taps8_odd_sizes", [(2, 121, 451, [0, 1], 96, 320)], "f32"),
    ("xfirst_scale_1p55", [(2, 149, 300, [1, 0], 96, 192)], "bf16"),
    ("yfirst_scale_1p65", [(2, 158, 300, [1, 0], 96, 192)], "bf16"),
    ("yfirst_near1_long_x", [(2, 64, 900, [0, 1], 64, 256)], "f32"),
    # x-first edges: a 5-pixel-wide source (windows run past the row into
    # the next row and past the frame's end), a source just wider than one
    # band, and eight open rows (2x vertical upscale) in fp32 with an odd
    # tap count
    ("xfirst_width5_source", [(3, 30, 5, [2, 0, 1], 32, 32)], "bf16"),
    ("xfirst_one_band_plus", [(2, 70, 67, [1, 0], 64, 64)], "f32"),
    ("xfirst_eight_slots_odd_taps", [(2, 48, 150, [0, 1], 96, 96)], "f32"),
    # targets taller than 2^15 rows (a unit's output rows beyond 16 bits):
    # one near 1 (x-first), one at 2x (y-first)
    ("tall_target_xfirst", [(2, 33000, 40, [1, 0], 32800, 32)], "bf16"),
    ("tall_target_yfirst", [(2, 66000, 48, [0, 1], 32800, 32)], "bf16"),
]


@pytest.mark.parametrize("name,specs,dtype", SMALL, ids=[s[0] for s in SMALL])
def test_small_cases_full(name, specs, dtype):
    mean, std = (0.481, 0.458, 0.408), (0.269, 0.261, 0.276)
    items, host = [], []
    for k, (n_src, H, W, idx, h, w) in enumerate(specs):
        it = _rand_video(100 + k, n_src, H, W)
        items.append((workloads.frames_torch(it, DEV), np.asarray(idx, np.int32), h, w))
        host.append(workloads.frames_np(it))
    log(f"case {name}: {[(s[0], s[1], s[2], s[4], s[5]) for s in specs]} {dtype}")
    out, grid, cu = run_gpu(items, mean, std, dtype)
    assert all_written(out)
    for k, (f, idx, h, w) in enumerate(items):
        ref = oracle.preprocess_item(host[k], idx, h, w, mean, std)
        assert_close(host_rows(out, cu[k], cu[k + 1], dtype), ref, dtype, f"{name} item {k}")


def _pairs_batch(items):
    """items padded with copies of the first until the plan takes column
    pairs; (batch, copies, launches)."""
    copies = 1
    while True:
        batch = items + [items[0]] * copies
        launches = vp.vp_batch_kernels([vp.Item(f, idx, h, w) for f, idx, h, w in batch])
        if any(r[0] == vp.VP_KERNEL_XFIRST and r[4] == 2 for r in launches):
            return batch, copies, launches
        copies *= 2
        assert copies <= 16384, "the plan never took column pairs"


# Column pairs on the x-first kernel (windows of 6 to 8 taps) are taken only
# in batches that give every wave slot four workgroups with single columns,
# so each case below is padded with copies of its first item (the same
# device frames) until the plan takes them; the distinct items are compared
# with the oracle in full, every copy with the first item's rows.
PAIRS = [
    # (name, [(n_src, H, W, indices, h, w)], dtype, x taps of the pair launches)
    ("pairs_480p_ragged_band", [(2, 480, 854, [1, 0], 320, 576)], "bf16", {6}),   # last band 64 of 128
    ("pairs_taps8_odd_sizes", [(2, 121, 611, [0, 1], 96, 320)], "f32", {8}),
    ("pairs_upscale_eight_slots", [(2, 48, 400, [0, 1], 96, 256)], "f32", {7}),
    # one band of 32 columns (16 lanes), windows past the row and the frame
    ("pairs_narrow_source", [(3, 40, 45, [2, 0, 1], 32, 32)], "bf16", {6}),
    # two pair shapes and a single-column item (5 taps) in one batch
    ("pairs_mixed", [(2, 150, 700, [1, 0], 96, 384), (2, 100, 500, [0, 1], 64, 288),
                     (2, 360, 640, [0, 1], 320, 576)], "bf16", {7, 8}),
]


@pytest.mark.parametrize("name,specs,dtype,pair_taps", PAIRS, ids=[s[0] for s in PAIRS])
def test_xfirst_column_pairs(name, specs, dtype, pair_taps):
    mean, std = (0.481, 0.458, 0.408), (0.269, 0.261, 0.276)
    items, host = [], []
    for k, (n_src, H, W, idx, h, w) in enumerate(specs):
        it = _rand_video(300 + k, n_src, H, W)
        items.append((workloads.frames_torch(it, DEV), np.asarray(idx, np.int32), h, w))
        host.append(workloads.frames_np(it))
    batch, copies, launches = _pairs_batch(items)
    paired = {int(r[2]) for r in launches if r[0] == vp.VP_KERNEL_XFIRST and r[4] == 2}
    assert paired == pair_taps, launches.tolist()
    log(f"case {name}: {len(specs)} items + {copies} copies, launches {launches.tolist()} {dtype}")
    out, grid, cu = run_gpu(batch, mean, std, dtype)
    assert all_written(out)
    for k, (f, idx, h, w) in enumerate(items):
        ref = oracle.preprocess_item(host[k], idx, h, w, mean, std)
        assert_close(host_rows(out, cu[k], cu[k + 1], dtype), ref, dtype, f"{name} item {k}")
    first = out[cu[0]:cu[1]]
    rest = out[cu[len(items)]:].view(copies, first.shape[0], first.shape[1])
    assert torch.equal(rest, first.unsqueeze(0).expand_as(rest)), "a copy differs from its original"


@pytest.mark.parametrize("case", range(8))
def test_xfirst_column_pairs_random(case):
    """Seeded random shapes for column pairs: vertical scales 0.5 to 1.6,
    horizontal 1.3 to 2 (6- to 8-tap windows), odd source sizes, unsorted
    indices with repeats and odd counts, fp32 and bf16."""
    rng = np.random.default_rng(7100 + case)
    dtype = "bf16" if case % 2 else "f32"
    mean, std = (0.481, 0.458, 0.408), (0.269, 0.261, 0.276)
    h = 32 * int(rng.integers(1, 8))
    w = 32 * int(rng.integers(1, 12))
    H = max(1, int(round(h * rng.uniform(0.5, 1.6)))) | 1
    W = int(round(w * rng.uniform(1.32, 1.95))) | 1
    n_src = int(rng.integers(1, 6))
    idx = rng.integers(0, n_src, size=int(rng.integers(1, 5))).astype(np.int32)
    it = _rand_video(500 + case, n_src, H, W)
    item = (workloads.frames_torch(it, DEV), idx, h, w)
    kx = vp.vp_filter_taps(W, w)
    if not 6 <= kx <= 8 or H > 1.6 * h:
        pytest.skip(f"drawn shape {H}x{W} -> {h}x{w} ({kx} taps) is not a column-pair shape")
    batch, copies, launches = _pairs_batch([item])
    log(f"pairs random {case}: {n_src}x{H}x{W} idx {idx.tolist()} -> {h}x{w} {dtype}, "
        f"{copies} copies, launches {launches.tolist()}")
    out, grid, cu = run_gpu(batch, mean, std, dtype)
    assert all_written(out)
    ref = oracle.preprocess_item(workloads.frames_np(it), idx, h, w, mean, std)
    assert_close(host_rows(out, cu[0], cu[1], dtype), ref, dtype, f"pairs random {case}")
    first = out[cu[0]:cu[1]]
    rest = out[cu[1]:].view(copies, first.shape[0], first.shape[1])
    assert torch.equal(rest, first.unsqueeze(0).expand_as(rest)), "a copy differs from its original"


def test_constant_frames_exact():
    f = torch.full((2, 77, 131, 3), 255, dtype=torch.uint8, device=DEV)
    out, _, _ = run_gpu([(f, np.array([0, 1], np.int32), 64, 96)], (0.5,) * 3, (0.5,) * 3, "bf16")
    bits = out.view(torch.int16).cpu().numpy().view(np.uint16)
    assert (bits == 0x3F80).all()          # exactly 1.0
    f.zero_()
    out, _, _ = run_gpu([(f, np.array([1], np.int32), 32, 32)], (0.5,) * 3, (0.5,) * 3, "f32")
    assert (out.cpu().numpy() == -1.0).all()


def test_identity_resize_is_the_normalised_input():
    it = _rand_video(7, 2, 96, 128)
    f = workloads.frames_torch(it, DEV)
    mean, std = (0.3, 0.4, 0.5), (0.2, 0.25, 0.3)
    out, _, _ = run_gpu([(f, np.array([1, 0], np.int32), 96, 128)], mean, std, "f32")
    v = out.cpu().numpy().reshape(1, 3, 4, 2, 2, 3, 2, 16, 16).transpose(0, 6, 5, 1, 3, 7, 2, 4, 8)
    v = v.reshape(2, 3, 96, 128)
    src = workloads.frames_np(it)[[1, 0]].transpose(0, 3, 1, 2).astype(np.float64)
    ref = (src / 255.0 - np.array(mean)[None, :, None, None]) / np.array(std)[None, :, None, None]
    assert np.abs(v - ref).max() <= 2e-5


def test_deterministic_and_on_side_stream():
    it = _rand_video(8, 4, 130, 170)
    f = workloads.frames_torch(it, DEV)
    items = [(f, np.array([0, 1, 2, 3], np.int32), 96, 128)]
    a, _, _ = run_gpu(items, (0.5,) * 3, (0.5,) * 3, "f32")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b, _, _ = run_gpu(items, (0.5,) * 3, (0.5,) * 3, "f32", stream=s)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# --------------------------------------------------------------------------
# the five workloads at full size
# --------------------------------------------------------------------------

def _materialise(wl):
    items, planned = [], []
    for it in wl.items:
        h, w, idx = plan_item(it)
        planned.append((h, w, idx))
        items.append((workloads.frames_torch(it, DEV), idx, h, w))
    return items, planned


THREADS = max(1, min(16, os.cpu_count() or 1))


def _padded(idx):
    return list(idx) + ([idx[-1]] if len(idx) % 2 else [])


def _check_pairs(out, cu, b, item_dev, idx, h, w, pairs, wl, dtype, patch=16, pool=None):
    """Whole frame pairs of item b against the oracle (frames copied from the
    device input), the oracle running in a thread pool.  Returns the merged
    comparison."""
    rows_per_t = (h // patch) * (w // patch)
    padded = _padded(idx)
    pairs = list(pairs)
    fids = sorted({padded[2 * tt + d] for tt in pairs for d in (0, 1)})
    pos = {f: k for k, f in enumerate(fids)}
    frames = item_dev[torch.as_tensor(fids, device=item_dev.device)].cpu().numpy()
    lo = cu[b] + min(pairs) * rows_per_t
    hi = cu[b] + (max(pairs) + 1) * rows_per_t
    gpu = host_rows(out, lo, hi, dtype)

    def one(tt):
        two = frames[[pos[padded[2 * tt]], pos[padded[2 * tt + 1]]]]
        ref = oracle.preprocess_item(two, [0, 1], h, w, wl.mean, wl.std, patch=patch)
        r0 = cu[b] + tt * rows_per_t - lo
        g = gpu[r0:r0 + rows_per_t]
        return compare.check_bf16(g, ref) if dtype == "bf16" else compare.check_f32(g, ref)

    own = pool is None
    pool = pool or cf.ThreadPoolExecutor(max_workers=THREADS)
    try:
        res = compare.merge(pool.map(one, pairs))
    finally:
        if own:
            pool.shutdown()
    return res


def _check_item_all(out, cu, b, item_dev, idx, h, w, wl, dtype, patch=16, pool=None):
    """Every row of item b, one frame pair per oracle call."""
    return _check_pairs(out, cu, b, item_dev, idx, h, w, range((len(idx) + 1) // 2), wl, dtype,
                        patch, pool)


def _check_sampled_rows(out, cu, b, item_dev, idx, h, w, rhos, wl, dtype, patch=16, pool=None):
    """Sampled rows of item b, each by the oracle's direct 2D sum (no
    separation into passes), in a thread pool.  Returns the merged comparison."""
    rows_per_t = (h // patch) * (w // patch)
    padded = _padded(idx)
    rhos = sorted(int(r) for r in rhos)
    pairs = sorted({r // rows_per_t for r in rhos})
    fids = sorted({padded[2 * tt + d] for tt in pairs for d in (0, 1)})
    pos = {f: k for k, f in enumerate(fids)}
    frames = item_dev[torch.as_tensor(fids, device=item_dev.device)].cpu().numpy()
    sel = torch.as_tensor([cu[b] + r for r in rhos], device=out.device)
    g = out.index_select(0, sel)
    gpu = g.view(torch.int16).cpu().numpy().view(np.uint16) if dtype == "bf16" else g.cpu().numpy()

    def one(k):
        rho = rhos[k]
        tt = rho // rows_per_t
        two = frames[[pos[padded[2 * tt]], pos[padded[2 * tt + 1]]]]
        return oracle.item_row(two, [0, 1], h, w, wl.mean, wl.std, rho - tt * rows_per_t, patch=patch)

    own = pool is None
    pool = pool or cf.ThreadPoolExecutor(max_workers=THREADS)
    try:
        refs = np.stack(list(pool.map(one, range(len(rhos)))))
    finally:
        if own:
            pool.shutdown()
    return compare.check_bf16(gpu, refs) if dtype == "bf16" else compare.check_f32(gpu, refs)


def _assert_res(res, what):
    log(f"{what}: {res}")
    assert res["ok"], f"{what}: {res}"


def test_workload_c0_full():
    wl = workloads.config(0)
    log(wl.name)
    items, _ = _materialise(wl)
    out, grid, cu = run_gpu(items, wl.mean, wl.std, wl.out_dtype)
    assert out.shape[0] == 320 and all_written(out)
    host = workloads.frames_np(wl.items[0])
    ref = oracle.preprocess_item(host, items[0][1], 128, 160, wl.mean, wl.std)
    assert_close(host_rows(out, 0, 320, "f32"), ref, "f32", "c0")


def test_workload_c1_full():
    wl = workloads.config(1)
    log(wl.name)
    items, planned = _materialise(wl)
    assert planned[0][:2] == (352, 640) and len(planned[0][2]) == 64
    out, grid, cu = run_gpu(items, wl.mean, wl.std, wl.out_dtype)
    assert out.shape[0] == 28160 and all_written(out)
    host = items[0][0].cpu().numpy()
    ref = oracle.preprocess_item(host, items[0][1], 352, 640, wl.mean, wl.std)
    assert_close(host_rows(out, 0, 28160, "f32"), ref, "f32", "c1 all rows")


def test_workload_c2_full_size():
    """128 frames of 1080x1920 -> 448x800, bf16: every one of the 89,600 rows."""
    wl = workloads.config(2)
    log(wl.name)
    items, _ = _materialise(wl)
    out, grid, cu = run_gpu(items, wl.mean, wl.std, wl.out_dtype)
    assert out.shape[0] == 89600 and all_written(out)
    f, idx, h, w = items[0]
    _assert_res(_check_item_all(out, cu, 0, f, idx, h, w, wl, "bf16"), "c2 all 89600 rows")


def test_workload_c3_full_size():
    """The ragged mixed batch (12 videos, 20 images), bf16: every row of every item."""
    wl = workloads.config(3)
    log(wl.name + f" ({len(wl.items)} items)")
    items, _ = _materialise(wl)
    out, grid, cu = run_gpu(items, wl.mean, wl.std, wl.out_dtype)
    assert all_written(out)
    results = []
    with cf.ThreadPoolExecutor(max_workers=THREADS) as pool:
        for b, (f, idx, h, w) in enumerate(items):
            results.append(_check_item_all(out, cu, b, f, idx, h, w, wl, "bf16", pool=pool))
    _assert_res(compare.merge(results), f"c3 all {int(cu[-1])} rows of {len(items)} items")


def test_workload_c4_full_size():
    """64 videos x 256 frames of 720x1280 (45.3 GB resident), in the launch
    configuration the benchmark times: one call, one stream.  Checked: eight
    whole videos (458,752 rows) against the separable oracle, and 100,352
    rows drawn from 16 frame pairs of every one of the 64 videos against the
    direct 2D sum."""
    wl = workloads.config(4)
    log(wl.name)
    items = []
    for it in wl.items:
        h, w, idx = plan_item(it)
        assert (h, w) == (256, 448)
        items.append((workloads.frames_torch(it, DEV, chunk=32), idx, h, w))
    log("c4 input generated")
    out, grid, cu = run_gpu(items, wl.mean, wl.std, wl.out_dtype)
    assert out.shape[0] == 3_670_016 and all_written(out)
    log("c4 ran; checking")
    # the device input equals the host generator on a few frames
    for b, fr in [(0, 0), (37, 255)]:
        assert np.array_equal(items[b][0][fr].cpu().numpy(),
                              workloads.frames_np(wl.items[b], [fr])[0])
    rng = np.random.default_rng(4)
    whole = sorted(set([0, 63]) | set(rng.choice(np.arange(1, 63), 6, replace=False).tolist()))
    rows_per_t = 16 * 28
    with cf.ThreadPoolExecutor(max_workers=THREADS) as pool:
        res = compare.merge(_check_item_all(out, cu, b, *items[b], wl, "bf16", pool=pool) for b in whole)
        _assert_res(res, f"c4 whole videos {whole}")
        sampled = []
        for b in range(64):   # 16 pairs x 98 rows per video: 100,352 rows in all
            pairs = rng.choice(128, 16, replace=False)
            rhos = (pairs[:, None] * rows_per_t + rng.integers(0, rows_per_t, (16, 98))).reshape(-1)
            sampled.append(_check_sampled_rows(out, cu, b, *items[b], rhos, wl, "bf16", pool=pool))
        res = compare.merge(sampled)
        assert res["n"] >= 100_000 * 1536
        _assert_res(res, "c4 sampled rows over all 64 videos")


# --------------------------------------------------------------------------
# Qwen2/2.5-VL geometry: patch 14 (windows of 28, rows of 1176)
# --------------------------------------------------------------------------

PATCH14 = [
    ("p14_downscale_f32", [(3, 150, 260, [2, 0], 84, 140)], "f32"),
    ("p14_upscale_bf16", [(2, 40, 50, [1, 0, 1], 56, 84)], "bf16"),
    ("p14_identity_f32", [(2, 56, 84, [1, 0], 56, 84)], "f32"),
    ("p14_ragged_bf16", [(5, 70, 90, [4, 1, 3], 56, 112), (1, 333, 257, [0], 308, 252),
                         (3, 480, 854, [0, 1, 2], 112, 196)], "bf16"),
    # an image and an odd count in fp32: one wave of the pair writes both
    # temporal halves of the (twice as large) stage
    ("p14_image_odd_f32", [(1, 333, 257, [0], 308, 252), (4, 150, 260, [3, 0, 2], 84, 140)], "f32"),
    ("p14_long_window", [(2, 540, 3840, [1, 0], 84, 672)], "bf16"),
    ("p14_taps10_px3", [(3, 180, 640, [0, 2], 84, 280)], "f32"),
    # items one band wide: the workgroup's second band is missing, and its
    # waves only keep step with the barriers (with an image in the batch,
    # whose pair is one frame twice)
    ("p14_single_band", [(2, 60, 70, [1, 0], 56, 56), (1, 40, 30, [0], 56, 28)], "bf16"),
]


@pytest.mark.parametrize("name,specs,dtype", PATCH14, ids=[c[0] for c in PATCH14])
def test_patch14_small_cases_full(name, specs, dtype):
    mean, std = (0.48145466, 0.4578275, 0.40821073), (0.26862954, 0.26130258, 0.27577711)
    items, host = [], []
    for k, (n_src, H, W, idx, h, w) in enumerate(specs):
        it = _rand_video(600 + k, n_src, H, W)
        items.append((workloads.frames_torch(it, DEV), np.asarray(idx, np.int32), h, w))
        host.append(workloads.frames_np(it))
    log(f"case {name}: {[(s[0], s[1], s[2], s[4], s[5]) for s in specs]} {dtype}")
    out, grid, cu = run_gpu(items, mean, std, dtype, patch=14)
    assert all_written(out)
    for k, (f, idx, h, w) in enumerate(items):
        ref = oracle.preprocess_item(host[k], idx, h, w, mean, std, patch=14)
        assert_close(host_rows(out, cu[k], cu[k + 1], dtype), ref, dtype, f"{name} item {k}")


def test_workload_q4_patch14_full_size():
    """Configuration 4's 64 x 256 frames in the patch-14 geometry (252x448,
    rows of 1176), in the launch configuration the benchmark times."""
    wl = workloads.patch14_config()
    log(wl.name)
    items = []
    for it in wl.items:
        h, w, idx = plan_item(it)
        assert (h, w) == (252, 448)
        items.append((workloads.frames_torch(it, DEV, chunk=32), idx, h, w))
    out, grid, cu = run_gpu(items, wl.mean, wl.std, wl.out_dtype, patch=14)
    assert out.shape[0] == 64 * 128 * 18 * 32 and all_written(out)
    rng = np.random.default_rng(14)
    rows_per_t = 18 * 32
    with cf.ThreadPoolExecutor(max_workers=THREADS) as pool:
        res = compare.merge(_check_item_all(out, cu, b, *items[b], wl, "bf16", patch=14, pool=pool)
                            for b in (0, 63))
        _assert_res(res, "q4 whole videos 0 and 63")
        sampled = []
        for b in range(64):   # 8 pairs x 40 rows per video
            pairs = rng.choice(128, 8, replace=False)
            rhos = (pairs[:, None] * rows_per_t + rng.integers(0, rows_per_t, (8, 40))).reshape(-1)
            sampled.append(_check_sampled_rows(out, cu, b, *items[b], rhos, wl, "bf16", patch=14, pool=pool))
        _assert_res(compare.merge(sampled), "q4 sampled rows over all 64 videos")

