"""CPU tests of the native library's host side: symbol exports, the host
planning functions bit-exact against the oracle, and every error path
(validation happens on the host before anything is enqueued, so no GPU is
needed)."""
import ctypes
import json
import os
import re

import numpy as np
import pytest

import oracle
import paper_2604_16893_amd as vp
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_function():
    header = open(os.path.join(ROOT, "include", "vp.h")).read()
    declared = set(re.findall(r"^\s*(?:int32_t|const char\*)\s+(vp_\w+)\s*\(", header, re.M))
    assert declared == set(vp.EXPORTED)
    L = ctypes.CDLL(vp.LIB_PATH)
    for name in declared:
        assert hasattr(L, name), name
    assert vp.lib().vp_status_string(vp.VP_ERR_CAPACITY) == b"VP_ERR_CAPACITY"


def test_smart_resize_bit_exact_vs_oracle():
    rng = np.random.default_rng(31)
    for _ in range(5000):
        H = int(rng.integers(1, 6000))
        W = int(rng.integers(1, 6000))
        B = int(rng.integers(1024, 9_000_000))
        mn = int(rng.integers(0, 2)) * int(rng.integers(0, B))
        try:
            want = oracle.smart_resize(H, W, 32, mn, B)
        except oracle.OracleError as e:
            with pytest.raises(vp.VPError) as got:
                vp.vp_smart_resize_dims(H, W, 32, mn, B)
            assert got.value.status == e.code
            continue
        assert vp.vp_smart_resize_dims(H, W, 32, mn, B) == want, (H, W, mn, B)


def test_sample_indices_bit_exact_vs_oracle():
    for N in range(1, 70):
        for n in range(1, N + 1):
            assert vp.vp_sample_indices(N, vp.VP_SAMPLE_UNIFORM, n).tolist() == \
                oracle.sample_uniform(N, n).tolist()
    rng = np.random.default_rng(32)
    for _ in range(2000):
        N = int(rng.integers(1, 20000))
        vf = float(rng.choice([23.976, 24.0, 25.0, 29.97, 30.0, 50.0, 60.0, 8.0, 1.0]))
        fps = float(rng.choice([0.5, 1.0, 2.0, 3.0, 4.0]))
        mn = int(rng.integers(1, 16))
        mx = int(rng.integers(mn, 800))
        try:
            want = oracle.sample_fps(N, vf, fps, mn, mx)
        except oracle.OracleError as e:
            with pytest.raises(vp.VPError) as got:
                vp.vp_sample_indices(N, vp.VP_SAMPLE_FPS, 0, vf, fps, mn, mx)
            assert got.value.status == e.code
            continue
        assert vp.vp_sample_indices(N, vp.VP_SAMPLE_FPS, 0, vf, fps, mn, mx).tolist() == \
            want.tolist()


def test_sample_indices_capacity_reports_count():
    L = vp.lib()
    cnt = ctypes.c_int32()
    out = (ctypes.c_int32 * 3)()
    st = L.vp_sample_indices(256, vp.VP_SAMPLE_FPS, 0, 8.0, 2.0, 4, 128, out, 3, ctypes.byref(cnt))
    assert st == vp.VP_ERR_CAPACITY and cnt.value == 64
    assert L.vp_sample_indices(10, 7, 3, 0, 0, 1, 1, out, 3, ctypes.byref(cnt)) == vp.VP_ERR_ARG
    assert L.vp_sample_indices(10, 0, 11, 0, 0, 1, 1, out, 3, ctypes.byref(cnt)) == vp.VP_ERR_FRAMES
    assert L.vp_sample_indices(10, 0, 3, 0, 0, 1, 1, out, 3, None) == vp.VP_ERR_NULL


AXES = [(320, 160), (240, 128), (854, 640), (480, 352), (1920, 800), (1080, 448), (1280, 448),
        (720, 256), (640, 576), (360, 320), (1280, 576), (720, 320), (10, 20), (7, 13),
        (300, 288), (1000, 32), (33, 32), (17, 64), (1024, 992), (256, 256), (3000, 96),
        (1, 32), (2, 64)]


@pytest.mark.parametrize("n_in,n_out", AXES)
def test_filter_table_matches_oracle(n_in, n_out):
    lo, cnt, w64 = oracle.filter_table(n_in, n_out)
    assert vp.vp_filter_taps(n_in, n_out) == w64.shape[1]
    start, count, w32 = vp.vp_filter_table(n_in, n_out)
    assert start.tolist() == lo.tolist() and count.tolist() == cnt.tolist()
    ref = w64.astype(np.float32)
    # computed in double and rounded once: within one float ulp of the oracle's
    # rounding; taps whose weight is exactly zero in exact arithmetic (the kernel
    # at |x| = 1 or 2) may carry double-rounding residue of order 1e-16
    tol = np.maximum(np.spacing(np.abs(ref)).astype(np.float64), 1e-15)
    assert np.all(np.abs(w32.astype(np.float64) - ref.astype(np.float64)) <= tol)


def _layout_items(k):
    wl = workloads.config(k)
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", "plan_configs.json")))
    g = gold["configs"][k]
    items = [vp.Item((0x10000, it["n_src"], it["H"], it["W"]), it["indices"], it["h"], it["w"])
             for it in g["items"]]
    return wl, g, items


@pytest.mark.parametrize("k", range(5))
def test_batch_layout_matches_golden_plan(k):
    wl, g, items = _layout_items(k)
    # dims from the library's own smart_resize agree with the oracle's fixture
    for it, gi in zip(wl.items, g["items"]):
        if it.dims is None:
            assert vp.vp_smart_resize_dims(it.H, it.W, 32, it.min_pixels, it.max_pixels) == \
                (gi["h"], gi["w"])
    grid, cu, rows, ws = vp.vp_batch_layout(items)
    assert grid.tolist() == g["grid_thw"]
    assert cu.tolist() == g["cu_seqlens"]
    assert rows == g["cu_seqlens"][-1]
    assert ws > 0 and ws % 256 == 0


def test_batch_layout_random_ragged_vs_oracle():
    rng = np.random.default_rng(33)
    for _ in range(50):
        B = int(rng.integers(1, 20))
        items, n_idx, hs, ws = [], [], [], []
        for _ in range(B):
            n_src = int(rng.integers(1, 40))
            n = int(rng.integers(1, n_src + 1))
            h = 32 * int(rng.integers(1, 20))
            w = 32 * int(rng.integers(1, 20))
            idx = rng.integers(0, n_src, size=n)
            items.append(vp.Item((0x10000, n_src, int(rng.integers(1, 999)),
                                  int(rng.integers(1, 999))), idx, h, w))
            n_idx.append(n)
            hs.append(h)
            ws.append(w)
        grid, cu, rows, _ = vp.vp_batch_layout(items)
        og, ocu = oracle.layout(n_idx, hs, ws)
        assert grid.tolist() == og.tolist() and cu.tolist() == ocu.tolist() and rows == ocu[-1]


def test_plan_cache_follows_every_field_and_index():
    """The library reuses the plan of an identical batch; any change of a
    field or an index (same frame buffer, same index array object mutated in
    place) must give that batch's own layout, including after eviction of
    older plans (more distinct batches than the cache holds)."""
    frames = (0x10000, 300, 720, 1280)
    idx = np.arange(0, 300, 2, dtype=np.int32)[:150]
    items = [vp.Item(frames, idx, 256, 448)]
    g1, cu1, r1, ws1 = vp.vp_batch_layout(items)
    idx[-1] = 299                          # same array, new content: same layout, new plan
    g2, cu2, r2, ws2 = vp.vp_batch_layout(items)
    assert (g1.tolist(), r1) == (g2.tolist(), r2)
    for k in range(12):                    # more distinct batches than the cache keeps
        n = 2 + 2 * k
        it = [vp.Item(frames, np.arange(n, dtype=np.int32), 256 - 32 * (k % 3), 448), items[0]]
        g, cu, rows, ws = vp.vp_batch_layout(it)
        og, ocu = oracle.layout([n, len(idx)], [256 - 32 * (k % 3), 256], [448, 448])
        assert g.tolist() == og.tolist() and cu.tolist() == ocu.tolist() and rows == ocu[-1]
    odd = [vp.Item(frames, idx[:149], 256, 448)]   # one index fewer: t = 75 either way
    g3, cu3, r3, _ = vp.vp_batch_layout(odd)
    assert g3.tolist() == [[75, 16, 28]] and r3 == r1
    # a bad index in a batch whose good twin was planned before is still reported
    bad = idx.copy()
    bad[5] = 300
    with pytest.raises(vp.VPError) as e:
        vp.vp_batch_layout([vp.Item(frames, bad, 256, 448)])
    assert e.value.status == vp.VP_ERR_INDEX


def test_layout_errors():
    ok = vp.Item((0x10000, 4, 100, 100), [0, 3], 64, 64)
    cases = [
        (vp.Item((0x10000, 4, 100, 100), [0, 4], 64, 64), vp.VP_ERR_INDEX),
        (vp.Item((0x10000, 4, 100, 100), [-1], 64, 64), vp.VP_ERR_INDEX),
        (vp.Item((0x10000, 4, 100, 100), [0], 48, 64), vp.VP_ERR_DIMS),
        (vp.Item((0x10000, 4, 100, 100), [0], 0, 64), vp.VP_ERR_DIMS),
        (vp.Item((0x10000, 4, 0, 100), [0], 64, 64), vp.VP_ERR_DIMS),
        (vp.Item((0x10000, 0, 100, 100), [0], 64, 64), vp.VP_ERR_FRAMES),
        (vp.Item((0x10000, 4, 100, 100), [], 64, 64), vp.VP_ERR_FRAMES),
        (vp.Item((0, 4, 100, 100), [0], 64, 64), vp.VP_ERR_NULL),
        (vp.Item((0x10000, 1, 40000, 40000), [0], 64, 64), vp.VP_ERR_CAPACITY),  # 4.8 GB frame
    ]
    for bad, code in cases:
        with pytest.raises(vp.VPError) as e:
            vp.vp_batch_layout([ok, bad])
        assert e.value.status == code, (bad, code)
    L = vp.lib()
    assert L.vp_batch_layout(None, 1, None, None, None, None) == vp.VP_ERR_NULL
    b = vp._Batch([ok])
    assert L.vp_batch_layout(b.arr, 0, None, None, None, None) == vp.VP_ERR_ARG


def _raw_preprocess(items, mean=(0.5,) * 3, std=(0.5,) * 3, dtype=vp.VP_OUT_BF16,
                    out=0x100000, cap=1 << 30, ws=0x200000, ws_bytes=1 << 30):
    b = vp._Batch(items)
    m = (ctypes.c_float * 3)(*mean)
    s = (ctypes.c_float * 3)(*std)
    return vp.lib().vp_preprocess_batch(b.arr, len(b), m, s, dtype, ctypes.c_void_p(out), cap,
                                        None, None, ctypes.c_void_p(ws), ws_bytes, None)


def test_preprocess_errors_before_any_gpu_work():
    """Every failure is detected on the host before the plan is uploaded."""
    ok = vp.Item((0x10000, 4, 100, 100), [0, 3], 64, 64)
    _, _, rows, need = vp.vp_batch_layout([ok])
    assert _raw_preprocess([ok], std=(0.5, 0.0, 0.5)) == vp.VP_ERR_ARG
    assert _raw_preprocess([ok], std=(0.5, -1.0, 0.5)) == vp.VP_ERR_ARG
    assert _raw_preprocess([ok], mean=(float("nan"), 0, 0)) == vp.VP_ERR_ARG
    assert _raw_preprocess([ok], dtype=5) == vp.VP_ERR_ARG
    assert _raw_preprocess([ok], out=0x100004) == vp.VP_ERR_ARG        # not 16-byte aligned
    assert _raw_preprocess([ok], ws=0x200010) == vp.VP_ERR_ARG         # not 256-byte aligned
    assert _raw_preprocess([ok], out=0) == vp.VP_ERR_NULL
    assert _raw_preprocess([ok], ws=0) == vp.VP_ERR_NULL
    assert _raw_preprocess([ok], cap=rows - 1) == vp.VP_ERR_CAPACITY
    assert _raw_preprocess([ok], ws_bytes=need - 1) == vp.VP_ERR_CAPACITY
    assert b"plan needs" in vp.lib().vp_last_error_message()
    assert _raw_preprocess([vp.Item((0x10000, 4, 100, 100), [9], 64, 64)]) == vp.VP_ERR_INDEX
    assert b"outside [0, 4)" in vp.lib().vp_last_error_message()


def _raw_noalloc(items, mean=(0.5, 0.5, 0.5), std=(0.5, 0.5, 0.5), dtype=vp.VP_OUT_BF16,
                 out=0x100000, cap=1 << 40):
    b = vp._Batch(items)
    m = (ctypes.c_float * 3)(*mean)
    s = (ctypes.c_float * 3)(*std)
    return vp.lib().vp_preprocess_batch_noalloc(b.arr, len(b), m, s, dtype, ctypes.c_void_p(out), cap,
                                                None, None, None)


def test_noalloc_errors_before_any_gpu_work():
    """The no-allocation entry checks everything on the host first, including
    that the plan fits the library's fixed plan memory (16 MiB), so these
    calls make no HIP call at all (none is possible here)."""
    ok = vp.Item((0x10000, 4, 100, 100), [0, 3], 64, 64)
    _, _, rows, _ = vp.vp_batch_layout([ok])
    assert _raw_noalloc([ok], std=(0.5, 0.0, 0.5)) == vp.VP_ERR_ARG
    assert _raw_noalloc([ok], dtype=5) == vp.VP_ERR_ARG
    assert _raw_noalloc([ok], out=0x100004) == vp.VP_ERR_ARG
    assert _raw_noalloc([ok], out=0) == vp.VP_ERR_NULL
    assert _raw_noalloc([ok], cap=rows - 1) == vp.VP_ERR_CAPACITY
    assert _raw_noalloc([vp.Item((0x10000, 4, 100, 100), [4], 64, 64)]) == vp.VP_ERR_INDEX
    # 262,144 frames of 720x1280 -> 256x448: one work unit and seven
    # workgroup entries per frame, a plan of about 11.5 MB -- within the limit;
    # twice as many frames need about 23 MB and are refused
    frames = (0x10000, 2, 720, 1280)
    small = [vp.Item(frames, [0, 1] * 2048, 256, 448) for _ in range(64)]
    big = small + small
    assert vp.vp_batch_layout(small)[3] <= vp.VP_NOALLOC_PLAN_BYTES < vp.vp_batch_layout(big)[3]
    assert _raw_noalloc(big) == vp.VP_ERR_CAPACITY
    assert b"fixed plan memory" in vp.lib().vp_last_error_message()


def _raw_patchify(items, mean=(0.5, 0.5, 0.5), std=(0.5, 0.5, 0.5), dtype=vp.VP_OUT_BF16,
                  out=0x100000, cap=1 << 30, ws=0x200000, ws_bytes=1 << 30):
    b = vp._Batch(items)
    m = (ctypes.c_float * 3)(*mean)
    s = (ctypes.c_float * 3)(*std)
    return vp.lib().vp_patchify_batch(b.arr, len(b), m, s, dtype, ctypes.c_void_p(out), cap,
                                      None, None, ctypes.c_void_p(ws), ws_bytes, None)


def test_patchify_errors_before_any_gpu_work():
    """The patchify-only entry takes frames already at the target size; every
    failure is detected on the host before anything is enqueued."""
    ok = vp.Item((0x10000, 4, 64, 96), [0, 3], 64, 96)
    _, _, rows, need = vp.vp_batch_layout([ok])
    assert _raw_patchify([vp.Item((0x10000, 4, 64, 96), [0, 3], 64, 64)]) == vp.VP_ERR_DIMS
    assert b"already at the target size" in vp.lib().vp_last_error_message()
    assert _raw_patchify([vp.Item((0x10000, 4, 60, 96), [0, 3], 60, 96)]) == vp.VP_ERR_DIMS
    assert _raw_patchify([vp.Item((0x10002, 4, 64, 96), [0, 3], 64, 96)]) == vp.VP_ERR_ARG
    assert b"4-byte aligned" in vp.lib().vp_last_error_message()
    assert _raw_patchify([vp.Item((0x10000, 4, 64, 96), [4], 64, 96)]) == vp.VP_ERR_INDEX
    assert _raw_patchify([ok], std=(0.5, 0.0, 0.5)) == vp.VP_ERR_ARG
    assert _raw_patchify([ok], dtype=7) == vp.VP_ERR_ARG
    assert _raw_patchify([ok], out=0x100008) == vp.VP_ERR_ARG
    assert _raw_patchify([ok], cap=rows - 1) == vp.VP_ERR_CAPACITY
    assert _raw_patchify([ok], ws_bytes=0) == vp.VP_ERR_CAPACITY
    assert _raw_patchify([ok], ws=0) == vp.VP_ERR_NULL
    # the layout of vp_batch_layout holds for this entry too: t = ceil(n_idx / 2)
    g, cu, rows3, _ = vp.vp_batch_layout([vp.Item((0x10000, 4, 64, 96), [0, 1, 2], 64, 96)])
    assert g.tolist() == [[2, 4, 6]] and rows3 == 48


def test_extreme_downscale_is_rejected_not_truncated():
    # a 40000-pixel-wide source to 32 columns: a horizontal window of ~5000
    # taps exceeds what the kernels stage; the call fails instead of clipping
    it = vp.Item((0x10000, 1, 100, 40000), [0], 32, 32)
    with pytest.raises(vp.VPError) as e:
        vp.vp_batch_layout([it])
    assert e.value.status == vp.VP_ERR_CAPACITY


@pytest.mark.parametrize("n_in,n_out", [(720, 256), (1280, 448), (1080, 448), (1920, 800),
                                         (480, 352), (854, 640), (40, 64), (96, 96),
                                         (3000, 96), (1, 32), (723, 736), (257, 256)])
def test_fixed_filter_table_bit_exact_vs_oracle(n_in, n_out):
    """The uint8 writer's 22-bit weights are rounded from the same doubles on
    both sides, so they agree bit for bit."""
    start, count, q = vp.vp_filter_table_fixed(n_in, n_out)
    for i in range(n_out):
        lo, ref = oracle.fixed_weights(n_in, n_out, i)
        assert start[i] == lo and count[i] == len(ref)
        assert np.array_equal(q[i, :count[i]], ref) and not q[i, count[i]:].any()


def test_resize_layout_offsets_and_errors():
    items = [vp.Item((0x10000, 5, 100, 70), [4, 0, 2], 64, 32),
             vp.Item((0x20000, 1, 40, 50), [0], 64, 96)]
    off, ws = vp.vp_resize_layout(items)
    assert off.tolist() == [0, 3 * 64 * 32 * 3, 3 * 64 * 32 * 3 + 64 * 96 * 3] and ws > 0
    L = vp.lib()
    b = vp._Batch(items)
    def raw(out=0x100000, cap=1 << 30, ws_ptr=0x200000, ws_bytes=1 << 30, its=b):
        return L.vp_resize_batch(its.arr, len(its), ctypes.c_void_p(out), cap, None,
                                 ctypes.c_void_p(ws_ptr), ws_bytes, None)
    assert raw(out=0x100002) == vp.VP_ERR_ARG          # output not 4-byte aligned
    assert raw(ws_ptr=0x200040) == vp.VP_ERR_ARG       # workspace not 256-byte aligned
    assert raw(out=0) == vp.VP_ERR_NULL
    assert raw(cap=int(off[-1]) - 1) == vp.VP_ERR_CAPACITY
    assert raw(ws_bytes=ws - 1) == vp.VP_ERR_CAPACITY
    assert raw(its=vp._Batch([vp.Item((0x10000, 5, 100, 70), [5], 64, 32)])) == vp.VP_ERR_INDEX
    assert raw(its=vp._Batch([vp.Item((0x10000, 5, 100, 70), [1], 60, 32)])) == vp.VP_ERR_DIMS
    # a window too long for any tile is rejected, not clipped
    with pytest.raises(vp.VPError) as e:
        vp.vp_resize_layout([vp.Item((0x10000, 1, 100, 40000), [0], 32, 32)])
    assert e.value.status == vp.VP_ERR_CAPACITY


def test_position_ids_segments_and_errors_on_host():
    """The ViT segments come back on the host; the device tables need a GPU
    (their errors are all found before anything is enqueued)."""
    items = [vp.Item((0x10000, 5, 100, 70), [4, 0, 2], 64, 32),
             vp.Item((0x20000, 1, 40, 50), [0], 96, 64)]
    L = vp.lib()
    b = vp._Batch(items)
    cu = np.zeros(4, np.int32)
    ns = ctypes.c_int32()
    ws = ctypes.c_void_p(0x200000)
    # no device table: only the segments, and nothing is enqueued
    assert L.vp_position_ids(b.arr, 2, None, None, 0, cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                             4, ctypes.byref(ns), ws, 1 << 20, None) == vp.VP_OK
    _, _, ocu = oracle.position_ids([3, 1], [64, 96], [32, 64])
    assert ns.value == 3 and cu.tolist() == ocu.tolist()
    cu_p = cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    assert L.vp_position_ids(b.arr, 2, None, None, 0, cu_p, 3, None, ws, 1 << 20, None) == vp.VP_ERR_CAPACITY
    dev = ctypes.c_void_p(0x300000)
    assert L.vp_position_ids(b.arr, 2, dev, None, 39, None, 0, None, ws, 1 << 20, None) == vp.VP_ERR_CAPACITY   # 40 rows
    assert L.vp_position_ids(b.arr, 2, ctypes.c_void_p(0x300002), None, 1 << 20, None, 0, None, ws,
                             1 << 20, None) == vp.VP_ERR_ARG
    assert L.vp_position_ids(b.arr, 2, dev, None, 1 << 20, None, 0, None, ctypes.c_void_p(0x200010),
                             1 << 20, None) == vp.VP_ERR_ARG
    assert L.vp_position_ids(b.arr, 2, dev, None, 1 << 20, None, 0, None, None, 1 << 20, None) == vp.VP_ERR_NULL
    bad = vp._Batch([vp.Item((0x10000, 5, 100, 70), [4, 0, 2], 64, 48)])
    assert L.vp_position_ids(bad.arr, 1, dev, None, 1 << 20, None, 0, None, ws, 1 << 20, None) == vp.VP_ERR_DIMS


def test_patch14_layout_and_checks():
    """Qwen2/2.5-VL geometry: patch 14, windows of 28, rows of 1176."""
    for H, W, maxp in [(720, 1280, 262144), (480, 854, 230400), (1024, 1024, 1003520), (720, 1280, 122880)]:
        assert vp.vp_smart_resize_dims(H, W, 28, 0, maxp) == oracle.smart_resize(H, W, 28, 0, maxp)
    items = [vp.Item((0x10000, 9, 100, 70), [4, 0, 2, 8, 1], 252, 448, patch=14),
             vp.Item((0x20000, 1, 40, 50), [0], 980, 980, patch=14)]
    grid, cu, rows, _ = vp.vp_batch_layout(items)
    og, ocu = oracle.layout([5, 1], [252, 980], [448, 980], patch=14)
    assert grid.tolist() == og.tolist() == [[3, 18, 32], [1, 70, 70]]
    assert cu.tolist() == ocu.tolist() and rows == cu[-1]
    assert vp.row_width(14) == 1176
    def status(its):
        with pytest.raises(vp.VPError) as e:
            vp.vp_batch_layout(its)
        return e.value.status
    assert status([vp.Item((0x10000, 2, 64, 64), [0], 64, 64, patch=14)]) == vp.VP_ERR_DIMS
    assert status([vp.Item((0x10000, 2, 64, 64), [0], 64, 64, patch=12)]) == vp.VP_ERR_ARG
    assert status([vp.Item((0x10000, 2, 64, 64), [0], 64, 64),
                   vp.Item((0x10000, 2, 64, 64), [0], 56, 56, patch=14)]) == vp.VP_ERR_ARG
    assert b"share one patch size" in vp.lib().vp_last_error_message()


def _workload_items(wl):
    """Items of a workload for the host-only entry points (frames are not read)."""
    out = []
    for it in wl.items:
        h, w = it.dims if it.dims is not None else vp.vp_smart_resize_dims(
            it.H, it.W, 2 * it.patch, it.min_pixels, it.max_pixels)
        s = it.sample
        idx = vp.vp_sample_indices(it.n_src, vp.VP_SAMPLE_UNIFORM, s["n"]) if s["mode"] == "uniform" else \
            vp.vp_sample_indices(it.n_src, vp.VP_SAMPLE_FPS, 0, s["video_fps"], s["fps"],
                                 s["min_frames"], s["max_frames"])
        out.append(vp.Item((1 << 20, it.n_src, it.H, it.W), idx, h, w, it.patch))
    return out


def test_batch_kernels_routes():
    """The launch description: x-first with single columns for the small
    480p batch, column pairs for the ragged batch's 6-tap (480p) videos only,
    the y-first kernel for strong downscales, and workgroup totals that add
    up to the plan's."""
    k1 = vp.vp_batch_kernels(_workload_items(workloads.config(1)))
    assert [tuple(r[:5]) for r in k1] == [(vp.VP_KERNEL_XFIRST, 5, 6, 0, 1)]
    k3 = vp.vp_batch_kernels(_workload_items(workloads.config(3)))
    xf = [r for r in k3 if r[0] == vp.VP_KERNEL_XFIRST]
    assert {int(r[2]) for r in xf if r[4] == 2} == {6}
    assert all(r[4] == 1 for r in xf if r[2] != 6)
    assert any(r[0] == vp.VP_KERNEL_YFIRST and r[2] == 9 for r in k3)
    k4 = vp.vp_batch_kernels(_workload_items(workloads.config(4)))
    assert [tuple(r) for r in k4] == [(vp.VP_KERNEL_YFIRST, 4, 12, 3, 0, 64 * 128 * 2 * 7)]
    n = ctypes.c_int32()
    assert vp.lib().vp_batch_kernels(None, 1, None, 0, None) == vp.VP_ERR_NULL
    assert vp.lib().vp_batch_kernels(None, 1, None, 1, ctypes.byref(n)) == vp.VP_ERR_ARG
    assert vp.lib().vp_batch_kernels(None, 1, None, 0, ctypes.byref(n)) == vp.VP_ERR_NULL   # items


def test_tall_targets_take_the_streaming_kernels():
    """Targets of 2^15 rows and more are planned like any other: the layout
    counts their rows, and they take the streaming kernels (their GPU parity
    is in tests/test_gpu_parity.py)."""
    for H, W, h, w, kind in ((33000, 40, 32800, 32, vp.VP_KERNEL_XFIRST),
                             (66000, 48, 32800, 32, vp.VP_KERNEL_YFIRST),
                             (131400, 48, 65600, 32, vp.VP_KERNEL_YFIRST)):
        items = [vp.Item((0x10000, 2, H, W), [0, 1], h, w)]
        grid, cu, rows, ws = vp.vp_batch_layout(items)
        assert grid.tolist() == [[1, h // 16, w // 16]] and rows == h // 16 * (w // 16)
        k = vp.vp_batch_kernels(items)
        assert [int(r[0]) for r in k] == [kind], k.tolist()


def test_batch_kernels_capacity_truncates():
    """With room for fewer rows than launches, vp_batch_kernels writes the
    first rows only and still reports the full count."""
    items = vp._Batch(_workload_items(workloads.config(3)))
    full = vp.vp_batch_kernels(_workload_items(workloads.config(3)))
    assert len(full) >= 3
    rows = np.full((3, 6), -7, np.int32)
    n = ctypes.c_int32()
    assert vp.lib().vp_batch_kernels(items.arr, len(items), vp._ptr(rows, ctypes.c_int32), 2,
                                     ctypes.byref(n)) == vp.VP_OK
    assert n.value == len(full)
    assert rows[:2].tolist() == full[:2].tolist() and (rows[2] == -7).all()
