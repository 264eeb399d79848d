"""Pins of the CPU oracle against values the mathematics fixes.

None of these re-types an oracle formula: each checks a closed form worked by
hand, an exact-arithmetic brute force, a library routine (fractions, numpy
matmul / reshape) or an invariant of the definition, chosen so that a dropped
term, a wrong sign or offset, or a transposed operand fails at least one.
References are to arXiv 2604.16893 (EasyVideoR1).
"""
import fractions
import math

import numpy as np
import pytest

import oracle

BIG = 1 << 62


# --------------------------------------------------------------------------
# smart_resize  (Section 3.1.1 resize under max_pixels; Section 3.1.2
# independent image / video budgets; Section 4.1 per-frame budget)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("H,W,minp,maxp,expect", [
    # worked by hand: rhe(15)=15, rhe(26.6875)=27 -> 480x864 > 230400;
    # beta = sqrt(409920/230400) = 1.33385; 480/beta/32 = 11.25 -> 352, 854/beta/32 = 20.01 -> 640
    (480, 854, 0, 230400, (352, 640)),
    # 360x640: 352x640 > 200704; beta = 15/14; 10.5 -> 10, 18.67 -> 18
    (360, 640, 0, 200704, (320, 576)),
    (480, 854, 0, 200704, (320, 576)),
    (720, 1280, 0, 200704, (320, 576)),
    # 1024^2 > 1003520; beta = 1.0222; 31.3 -> 31
    (1024, 1024, 0, 1003520, (992, 992)),
    (256, 256, 0, 1003520, (256, 256)),
    (1080, 1920, 0, 368640, (448, 800)),
    (720, 1280, 0, 122880, (256, 448)),
    (240, 320, 0, 24576, (128, 160)),
    # no budget: rhe(7.5) = 8, rhe(10) = 10
    (240, 320, 0, BIG, (256, 320)),
    # rhe(22.5) = 22 (half to even, not half up) -- pins the tie rule
    (720, 1280, 0, BIG, (704, 1280)),
    # the paper's own budgets (Section 4.1): beta = 15/8 and 45/16 exactly
    (720, 1280, 0, 262144, (384, 672)),
    (1080, 1920, 0, 262144, (384, 672)),
    (1024, 1024, 0, 1048576, (1024, 1024)),
    # min branch: rhe(1.5625)=2, rhe(2.5)=2 -> 64x64 < 65536; beta = sqrt(16.384)
    # = 4.0477; ceil(6.32) = 7 -> 224, ceil(10.12) = 11 -> 352
    (50, 80, 65536, BIG, (224, 352)),
    # factor clamp: a 20-pixel side rounds to 32
    (20, 300, 0, BIG, (32, 288)),
])
def test_smart_resize_worked_values(H, W, minp, maxp, expect):
    assert oracle.smart_resize(H, W, 32, minp, maxp) == expect


def test_smart_resize_errors():
    with pytest.raises(oracle.OracleError) as e:
        oracle.smart_resize(10, 2001, 32, 0, BIG)       # ratio 200.1 > 200
    assert e.value.code == oracle.ERR_ASPECT
    # ratio exactly 200 is allowed; 2000/32 = 62.5 rounds half to even to 62
    assert oracle.smart_resize(10, 2000, 32, 0, BIG) == (32, 1984)
    for bad in [(0, 10), (10, 0), (-5, 10)]:
        with pytest.raises(oracle.OracleError) as e:
            oracle.smart_resize(bad[0], bad[1], 32, 0, BIG)
        assert e.value.code == oracle.ERR_ARG
    with pytest.raises(oracle.OracleError):
        oracle.smart_resize(100, 100, 32, 1000, 10)     # min > max
    with pytest.raises(oracle.OracleError):
        oracle.smart_resize(100, 100, 32, 0, 0)


def _kmax_exact(H, W, B, F):
    """Largest k >= 0 with (k F)^2 W <= H B: the exact value of floor(H / beta / F)."""
    k = math.isqrt(H * B // W) // F + 2
    while k > 0 and (k * F) ** 2 * W > H * B:
        k -= 1
    return k


def test_smart_resize_max_branch_matches_exact_arithmetic():
    """floor(H / sqrt(H W / B) / F) equals the exact-integer answer except at
    near-exact boundaries, where the double-precision sequence decides."""
    rng = np.random.default_rng(11)
    checked = 0
    for _ in range(4000):
        H = int(rng.integers(32, 4000))
        W = int(rng.integers(32, 4000))
        if max(H, W) / min(H, W) > 200:
            continue
        B = int(rng.integers(32 * 32, 4_000_000))
        h, w = oracle.smart_resize(H, W, 32, 0, B)
        h0 = max(32, round(H / 32) * 32)
        w0 = max(32, round(W / 32) * 32)
        if h0 * w0 <= B:
            assert (h, w) == (h0, w0)
            continue
        for got, A, Bo in ((h, H, W), (w, W, H)):
            k = _kmax_exact(A, Bo, B, 32)
            exact_q = math.sqrt(A * B / Bo) / 32
            if abs(exact_q - round(exact_q)) > 1e-9:
                assert got == max(32, 32 * k), (H, W, B)
        checked += 1
    assert checked > 1000


def test_smart_resize_invariants_and_idempotence():
    """Multiples of 32, within budget, and stage-consistent: re-running on
    the already-resized size returns the same size (Section 3.1.1: every
    stage must produce identical video_grid_thw)."""
    rng = np.random.default_rng(12)
    for _ in range(3000):
        H = int(rng.integers(1, 5000))
        W = int(rng.integers(1, 5000))
        if max(H, W) / min(H, W) > 200:
            continue
        B = int(rng.integers(32 * 32 * 4, 3_000_000))
        h, w = oracle.smart_resize(H, W, 32, 0, B)
        assert h % 32 == 0 and w % 32 == 0 and h >= 32 and w >= 32
        if h > 32 and w > 32:
            assert h * w <= B
            assert oracle.smart_resize(h, w, 32, 0, B) == (h, w)


# --------------------------------------------------------------------------
# Frame-index sampling (Section 3.1.1 cache key (path, fps, max_frames,
# max_pixels); Section 4.1 "2 FPS with a maximum of 128 frames")
# --------------------------------------------------------------------------

def test_uniform_indices_worked_values():
    # i * 15 / 7 = 0, 2.14, 4.29, 6.43, 8.57, 10.71, 12.86, 15
    assert oracle.sample_uniform(16, 8).tolist() == [0, 2, 4, 6, 9, 11, 13, 15]
    # N=30, n=15, i=7: 7 * 29 / 14 = 14.5 exactly -> half to even -> 14
    assert oracle.sample_uniform(30, 15)[7] == 14
    assert oracle.sample_uniform(30, 15)[1] == 2      # 29/14 = 2.07
    assert oracle.sample_uniform(5, 1).tolist() == [0]
    assert oracle.sample_uniform(256, 256).tolist() == list(range(256))
    c2 = oracle.sample_uniform(512, 128)
    assert c2[:10].tolist() == [0, 4, 8, 12, 16, 20, 24, 28, 32, 36]
    assert c2[-1] == 511


def test_uniform_indices_brute_force_fractions():
    """Python's round() on an exact Fraction rounds half to even."""
    for N in range(1, 61):
        for n in range(1, N + 1):
            got = oracle.sample_uniform(N, n).tolist()
            if n == 1:
                want = [0]
            else:
                want = [round(fractions.Fraction(i * (N - 1), n - 1)) for i in range(n)]
            assert got == want, (N, n)
            assert got[0] == 0
            if n >= 2:
                assert got[-1] == N - 1
            assert all(b > a for a, b in zip(got, got[1:]))


def test_uniform_indices_errors():
    for N, n in [(4, 5), (4, 0), (0, 1)]:
        with pytest.raises(oracle.OracleError) as e:
            oracle.sample_uniform(N, n)
        assert e.value.code == oracle.ERR_FRAMES


def test_fps_indices():
    # 256 frames at 8 fps resampled at 2 fps: 64 frames, i * 255 / 63
    idx = oracle.sample_fps(256, 8.0, 2.0, 4, 128)
    assert len(idx) == 64
    assert idx[:16].tolist() == [0, 4, 8, 12, 16, 20, 24, 28, 32, 36, 40, 45, 49, 53, 57, 61]
    assert idx[-4:].tolist() == [243, 247, 251, 255]
    # 7 frames at 1 fps -> 7 -> even 6: i * 6 / 5 = 0, 1.2, 2.4, 3.6, 4.8, 6
    assert oracle.sample_fps(7, 1.0, 1.0, 2, 100).tolist() == [0, 1, 2, 4, 5, 6]
    # a 10-minute clip at 30 fps sampled at 2 fps is capped at 128 frames (Section 4.1)
    long_clip = oracle.sample_fps(18000, 30.0, 2.0, 4, 128)
    assert len(long_clip) == 128 and long_clip[-1] == 17999
    # min_frames raises a short clip's count: 20 frames at 30 fps @2fps -> 1.33 -> 4
    assert len(oracle.sample_fps(20, 30.0, 2.0, 4, 128)) == 4
    # odd max_frames floors to even
    assert len(oracle.sample_fps(1000, 1.0, 1.0, 4, 255)) == 254
    with pytest.raises(oracle.OracleError) as e:
        oracle.sample_fps(1, 30.0, 2.0, 1, 10)
    assert e.value.code == oracle.ERR_FRAMES


# --------------------------------------------------------------------------
# Keys cubic kernel and antialiased filter weights
# --------------------------------------------------------------------------

def test_keys_kernel_values():
    # a = -0.5: K(0.25) = 1.5/64 - 2.5/16 + 1 = 0.8671875; K(0.75) = 0.2265625;
    # K(1.25) = -0.5*1.953125 + 2.5*1.5625 - 5 + 2 = -0.0703125; K(1.75) = -0.0234375
    for x, v in [(0.0, 1.0), (0.25, 0.8671875), (0.75, 0.2265625), (1.0, 0.0),
                 (1.25, -0.0703125), (1.75, -0.0234375), (2.0, 0.0), (2.5, 0.0), (0.5, 0.5625),
                 (1.5, -0.0625)]:
        assert oracle.keys_cubic(x) == v
        assert oracle.keys_cubic(-x) == v


def test_keys_kernel_reproduces_quadratics():
    """Keys' a = -1/2 kernel interpolates polynomials of degree <= 2 exactly:
    sum_k K(t - k) p(k) = p(t)."""
    rng = np.random.default_rng(5)
    for t in rng.uniform(-3, 3, 50):
        ks = range(math.floor(t) - 2, math.floor(t) + 3)
        for p in (lambda u: 1.0, lambda u: u, lambda u: 3 * u * u - u + 2):
            s = sum(oracle.keys_cubic(t - k) * p(k) for k in ks)
            assert abs(s - p(t)) < 1e-12


def test_filter_exact_2x_downscale_interior():
    # 320 -> 160, output 40: centre 81, taps j = 77..84 at (j + 0.5 - 81)/2 =
    # -1.75 .. 1.75; the raw sum is 2, so weights are K/2
    lo, w = oracle.filter_weights(320, 160, 40)
    assert lo == 77
    assert w.tolist() == [-0.01171875, -0.03515625, 0.11328125, 0.43359375,
                          0.43359375, 0.11328125, -0.03515625, -0.01171875]


def test_filter_exact_2x_downscale_border_renormalised():
    # output 0: centre 1, window [max(0, -3), 5): K(-0.25), K(0.25), K(0.75), K(1.25), K(1.75)
    lo, w = oracle.filter_weights(320, 160, 0)
    raw = np.array([0.8671875, 0.8671875, 0.2265625, -0.0703125, -0.0234375])
    assert lo == 0
    np.testing.assert_allclose(w, raw / 1.8671875, rtol=0, atol=1e-16)


def test_filter_exact_2x_upscale():
    # 10 -> 20, output i = 2m: centre m + 0.25, window [m - 2, m + 2),
    # offsets -1.75, -0.75, 0.25, 1.25; raw sum 1 (no renormalisation)
    lo, w = oracle.filter_weights(10, 20, 8)
    assert lo == 2
    assert w.tolist() == [-0.0234375, 0.2265625, 0.8671875, -0.0703125]
    # odd output i = 2m + 1: centre m + 0.75, window [m - 1, m + 3), mirrored weights
    lo, w = oracle.filter_weights(10, 20, 9)
    assert lo == 3
    assert w.tolist() == [-0.0703125, 0.8671875, 0.2265625, -0.0234375]


def test_filter_identity():
    # s = 1: centre i + 0.5, window [i - 1, i + 3), offsets -1, 0, 1, 2
    for i in range(1, 7):
        lo, w = oracle.filter_weights(10, 10, i)
        assert lo == i - 1
        assert w.tolist() == [0.0, 1.0, 0.0, 0.0]


@pytest.mark.parametrize("n_in,n_out", [(320, 160), (240, 128), (854, 640), (480, 352),
                                        (1920, 800), (1080, 448), (1280, 448), (720, 256),
                                        (640, 576), (360, 320), (10, 20), (7, 13), (300, 288),
                                        (1000, 32), (33, 32), (17, 64)])
def test_filter_sum_one_and_mirror_symmetry(n_in, n_out):
    lo, cnt, w = oracle.filter_table(n_in, n_out)
    for i in range(n_out):
        assert abs(w[i, :cnt[i]].sum() - 1.0) < 1e-13
        assert 0 <= lo[i] and lo[i] + cnt[i] <= n_in
    # mirror: w(n_out-1-i, n_in-1-j) = w(i, j), up to zero-weight edge taps
    dense = np.zeros((n_out, n_in))
    for i in range(n_out):
        dense[i, lo[i]:lo[i] + cnt[i]] = w[i, :cnt[i]]
    np.testing.assert_allclose(dense[::-1, ::-1], dense, rtol=0, atol=1e-13)


def test_filter_max_taps_of_workload_axes():
    """Longest windows: about 4 * sigma + 1 taps (support 2 sigma each side)."""
    for n_in, n_out, k in [(320, 160, 8), (240, 128, 8), (854, 640, 6), (480, 352, 6),
                           (1920, 800, 10), (1080, 448, 10), (1280, 448, 12), (720, 256, 12),
                           (640, 576, 5), (1280, 576, 9), (100, 300, 4)]:
        assert oracle.filter_table(n_in, n_out)[2].shape[1] == k, (n_in, n_out)


# --------------------------------------------------------------------------
# Resampling of a frame
# --------------------------------------------------------------------------

def _rand_frame(rng, H, W):
    return rng.integers(0, 256, size=(H, W, 3), dtype=np.uint8)


def test_resize_identity_is_exact():
    rng = np.random.default_rng(1)
    f = _rand_frame(rng, 37, 53)
    r = oracle.resize_frame(f, 37, 53)
    assert np.array_equal(r, f.transpose(2, 0, 1).astype(np.float64))


def test_resize_constant_frame():
    for (H, W, h, w) in [(40, 60, 32, 32), (20, 30, 64, 96), (720, 1280, 32, 64)]:
        f = np.full((H, W, 3), 173, np.uint8)
        r = oracle.resize_frame(f, h, w)
        np.testing.assert_allclose(r, 173.0, rtol=0, atol=1e-11)


@pytest.mark.parametrize("H,W,h,w", [(7, 9, 4, 5), (5, 6, 11, 13), (33, 47, 32, 32),
                                     (64, 40, 32, 64), (12, 90, 12, 7)])
def test_resize_separable_equals_direct_2d_sum(H, W, h, w):
    rng = np.random.default_rng(H * 1000 + W)
    f = _rand_frame(rng, H, W)
    r = oracle.resize_frame(f, h, w)
    for c in range(3):
        for i in range(h):
            for j in range(w):
                assert abs(r[c, i, j] - oracle.resize_pixel(f, h, w, i, j, c)) < 1e-10


@pytest.mark.parametrize("H,W,h,w", [(48, 80, 32, 32), (30, 20, 64, 96), (100, 71, 64, 32)])
def test_resize_equals_dense_matrix_product(H, W, h, w):
    """R_c = Wy F_c Wx^T with dense weight matrices (numpy matmul)."""
    rng = np.random.default_rng(7)
    f = _rand_frame(rng, H, W)
    r = oracle.resize_frame(f, h, w)

    def dense(n_in, n_out):
        lo, cnt, wt = oracle.filter_table(n_in, n_out)
        m = np.zeros((n_out, n_in))
        for i in range(n_out):
            m[i, lo[i]:lo[i] + cnt[i]] = wt[i, :cnt[i]]
        return m
    Wy, Wx = dense(H, h), dense(W, w)
    for c in range(3):
        np.testing.assert_allclose(r[c], Wy @ f[:, :, c].astype(np.float64) @ Wx.T,
                                   rtol=0, atol=1e-10)


def test_resize_flip_equivariance_and_linearity():
    rng = np.random.default_rng(9)
    f = rng.integers(0, 128, size=(45, 70, 3), dtype=np.uint8)
    g = rng.integers(0, 128, size=(45, 70, 3), dtype=np.uint8)
    r = oracle.resize_frame(f, 32, 32)
    np.testing.assert_allclose(oracle.resize_frame(f[:, ::-1], 32, 32), r[:, :, ::-1], atol=1e-10)
    np.testing.assert_allclose(oracle.resize_frame(f[::-1], 32, 32), r[:, ::-1], atol=1e-10)
    np.testing.assert_allclose(oracle.resize_frame(f + g, 32, 32),
                               r + oracle.resize_frame(g, 32, 32), atol=1e-10)


def test_resize_upscale_reproduces_quadratic_of_pixel_centres():
    """Pixel j of the source carries p(j + 0.5) with p(t) = 4 t^2 (integers
    4 j^2 + 4 j + 1).  Upscaled output i samples the continuous coordinate
    (i + 0.5) * s; where its window is not cut by a border, the value is
    p((i + 0.5) * s) exactly.  Pins the half-pixel convention, the kernel
    orientation and the scale."""
    W, w = 8, 20
    row = np.array([4 * j * j + 4 * j + 1 for j in range(W)], np.uint8)
    f = np.broadcast_to(row[None, :, None], (4, W, 3)).copy()
    r = oracle.resize_frame(f, 4, w)
    s = W / w
    for i in range(w):
        c = (i + 0.5) * s
        if c - 1.5 >= 0 and c + 2.5 <= W:
            assert abs(r[0, 1, i] - 4 * c * c) < 1e-9, i


def test_resize_2x_downscale_reproduces_linear_ramp():
    """Symmetric exact-2x weights reproduce a linear function of the pixel
    centre: value 2 j at centre j + 0.5 gives 2 * (2 i + 1) - 1 at output i."""
    H, W = 40, 64
    f = np.broadcast_to((2 * np.arange(H, dtype=np.uint8))[:, None, None], (H, W, 3)).copy()
    r = oracle.resize_frame(f, 20, 32)
    for i in range(2, 18):
        assert abs(r[1, i, 5] - (2 * (2 * i + 1) - 1)) < 1e-10


def test_resize_ringing_bound():
    """|R| stays within 255 * (L +- 1) / 2 with L the product of the two axes'
    absolute weight sums."""
    f = np.zeros((30, 30, 3), np.uint8)
    f[:, 15:] = 255
    r = oracle.resize_frame(f, 64, 64)
    _, cy, wy = oracle.filter_table(30, 64)
    _, cx, wx = oracle.filter_table(30, 64)
    L = np.abs(wy).sum(1)[:, None] * np.abs(wx).sum(1)[None, :]
    assert (r[0] >= -255 * (L - 1) / 2 - 1e-9).all() and (r[0] <= 255 * (L + 1) / 2 + 1e-9).all()
    assert r.min() < 0 and r.max() > 255      # bicubic ringing is kept, not clamped


# --------------------------------------------------------------------------
# Normalisation, padding, patchify, grid_thw / cu_seqlens
# --------------------------------------------------------------------------

def test_normalize_constants():
    assert oracle.normalize(255.0, 0.5, 0.5) == 1.0
    assert oracle.normalize(0.0, 0.5, 0.5) == -1.0
    f = np.full((2, 64, 64, 3), 255, np.uint8)
    rows = oracle.preprocess_item(f, [0, 1], 32, 32, (0.5,) * 3, (0.5,) * 3)
    assert np.all(np.abs(rows - 1.0) < 1e-12)
    f[:] = 51
    m, s = (0.481, 0.458, 0.408), (0.269, 0.261, 0.276)
    rows = oracle.preprocess_item(f, [1, 0], 32, 32, m, s)
    for c in range(3):
        np.testing.assert_allclose(rows[:, 512 * c:512 * (c + 1)], (0.2 - m[c]) / s[c], atol=1e-12)


def _identity_item(values):
    """Frames with the given per-(frame, channel, y, x) uint8 values."""
    return np.ascontiguousarray(values.transpose(0, 2, 3, 1)).astype(np.uint8)


def test_patchify_row_and_column_order():
    # 2 frames, 32 x 96: grid (1, 2, 6); merge windows (bh, bw) in raster order
    H, W = 32, 96
    vals = np.zeros((2, 3, H, W), np.int64)
    ii, jj = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    vals[:, 0] = 10 * (ii // 16) + (jj // 16)           # patch id in channel 0
    for fr in range(2):
        vals[fr, 1] = 50 + 10 * fr                      # (ch, dt) code in channel 1
        vals[fr, 2] = 16 * (ii % 16) + (jj % 16)        # raster position in channel 2
    f = _identity_item(vals)
    rows = oracle.preprocess_item(f, [0, 1], H, W, (0.0,) * 3, (1 / 255,) * 3)
    assert rows.shape == (12, 1536)
    patch = np.rint(rows[:, :256].mean(1)).astype(int).tolist()
    # rows 0..3 are patches (0,0),(0,1),(1,0),(1,1); row 4 is (0,2); row 8 is (0,4)
    assert patch == [0, 1, 10, 11, 2, 3, 12, 13, 4, 5, 14, 15]
    # column blocks: (ch, dt) = (1, 0) at 512, (1, 1) at 768
    assert np.allclose(rows[:, 512:768], 50) and np.allclose(rows[:, 768:1024], 60)
    # raster order inside a 16 x 16 patch: column 1024 + 16 y + x holds 16 y + x
    assert np.allclose(rows[:, 1024:1280], np.arange(256)[None, :])
    assert np.allclose(rows[:, 1280:1536], np.arange(256)[None, :])


def test_patchify_inverse_by_reshape():
    """Undoing the merge-window order with numpy reshape/transpose restores
    the normalised frames exactly (identity resize)."""
    rng = np.random.default_rng(21)
    n, H, W = 4, 64, 96
    f = rng.integers(0, 256, size=(n, H, W, 3), dtype=np.uint8)
    mean, std = (0.3, 0.4, 0.5), (0.2, 0.25, 0.3)
    idx = [3, 0, 2, 1]
    rows = oracle.preprocess_item(f, idx, H, W, mean, std)
    t, hm, wm = 2, H // 32, W // 32
    v = rows.reshape(t, hm, wm, 2, 2, 3, 2, 16, 16)          # tt bh bw mh mw c dt y x
    v = v.transpose(0, 6, 5, 1, 3, 7, 2, 4, 8)               # tt dt c bh mh y bw mw x
    v = v.reshape(2 * t, 3, H, W)
    ref = (f[idx].transpose(0, 3, 1, 2) / 255.0 - np.array(mean)[None, :, None, None]) \
        / np.array(std)[None, :, None, None]
    np.testing.assert_allclose(v, ref, rtol=0, atol=1e-12)


def test_image_is_duplicated_and_odd_count_padded():
    rng = np.random.default_rng(22)
    f = rng.integers(0, 256, size=(3, 40, 70, 3), dtype=np.uint8)
    rows = oracle.preprocess_item(f, [2], 32, 64, (0.5,) * 3, (0.5,) * 3)
    assert rows.shape == (8, 1536)
    for c in range(3):
        assert np.array_equal(rows[:, 512 * c:512 * c + 256], rows[:, 512 * c + 256:512 * c + 512])
    # three indices -> padded to four with the last one repeated
    r3 = oracle.preprocess_item(f, [0, 1, 2], 32, 64, (0.5,) * 3, (0.5,) * 3)
    r4 = oracle.preprocess_item(f, [0, 1, 2, 2], 32, 64, (0.5,) * 3, (0.5,) * 3)
    assert np.array_equal(r3, r4)


def test_item_row_direct_equals_separable_rows():
    rng = np.random.default_rng(23)
    f = rng.integers(0, 256, size=(5, 50, 90, 3), dtype=np.uint8)
    idx, mean, std = [4, 1, 3], (0.48, 0.46, 0.41), (0.27, 0.26, 0.28)
    rows = oracle.preprocess_item(f, idx, 64, 96, mean, std)
    for rho in [0, 1, 5, 11, 12, 23, rows.shape[0] - 1]:
        np.testing.assert_allclose(oracle.item_row(f, idx, 64, 96, mean, std, rho), rows[rho],
                                   rtol=0, atol=1e-12)


def test_row_counts_and_layout():
    assert oracle.item_rows(8, 128, 160) == 320          # 4 x 8 x 10
    assert oracle.item_rows(64, 352, 640) == 28160       # 32 x 22 x 40
    assert oracle.item_rows(128, 448, 800) == 89600      # 64 x 28 x 50
    assert oracle.item_rows(256, 256, 448) == 57344      # 128 x 16 x 28
    assert oracle.item_rows(1, 992, 992) == 3844         # t = 1 for an image
    g, cu = oracle.layout([8, 1, 3], [128, 992, 64], [160, 992, 32])
    assert g.tolist() == [[4, 8, 10], [1, 62, 62], [2, 4, 2]]
    assert cu.tolist() == [0, 320, 320 + 3844, 320 + 3844 + 16]
    g, cu = oracle.layout([256] * 64, [256] * 64, [448] * 64)
    assert cu[-1] == 3_670_016


def test_errors_of_item_checks():
    f = np.zeros((2, 40, 40, 3), np.uint8)
    with pytest.raises(oracle.OracleError) as e:
        oracle.preprocess_item(f, [0, 2], 32, 32, (0.5,) * 3, (0.5,) * 3)
    assert e.value.code == oracle.ERR_INDEX
    with pytest.raises(oracle.OracleError) as e:
        oracle.preprocess_item(f, [0, 1], 32, 48, (0.5,) * 3, (0.5,) * 3)
    assert e.value.code == oracle.ERR_DIMS


# -- normalise + patchify only (frames already at the target size) --------

def test_patchify_only_inverse_by_reshape():
    """Undoing the merge-window order of the patchify-only path with numpy
    reshape/transpose gives the normalised, padded frames bit for bit."""
    rng = np.random.default_rng(31)
    n, h, w = 5, 64, 96
    f = rng.integers(0, 256, size=(n, h, w, 3), dtype=np.uint8)
    mean, std = (0.481, 0.458, 0.408), (0.269, 0.261, 0.276)
    idx = [4, 0, 2]                                           # odd: padded with 2
    rows = oracle.patchify_item(f, idx, mean, std)
    t, hm, wm = 2, h // 32, w // 32
    assert rows.shape == (t * hm * wm * 4, 1536)
    v = rows.reshape(t, hm, wm, 2, 2, 3, 2, 16, 16)           # tt bh bw mh mw c dt y x
    v = v.transpose(0, 6, 5, 1, 3, 7, 2, 4, 8).reshape(2 * t, 3, h, w)
    ref = (f[[4, 0, 2, 2]].transpose(0, 3, 1, 2) / 255.0 - np.array(mean)[None, :, None, None]) \
        / np.array(std)[None, :, None, None]
    assert np.array_equal(v, ref)


def test_patchify_only_row_and_column_order():
    # the planted codes of the full path's order test, read back through the
    # patchify-only path
    H, W = 32, 96
    vals = np.zeros((2, 3, H, W), np.int64)
    ii, jj = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    vals[:, 0] = 10 * (ii // 16) + (jj // 16)
    for fr in range(2):
        vals[fr, 1] = 50 + 10 * fr
        vals[fr, 2] = 16 * (ii % 16) + (jj % 16)
    f = _identity_item(vals)
    rows = oracle.patchify_item(f, [0, 1], (0.0,) * 3, (1 / 255,) * 3)
    patch = np.rint(rows[:, :256].mean(1)).astype(int).tolist()
    assert patch == [0, 1, 10, 11, 2, 3, 12, 13, 4, 5, 14, 15]
    assert np.allclose(rows[:, 512:768], 50) and np.allclose(rows[:, 768:1024], 60)
    assert np.allclose(rows[:, 1024:1280], np.arange(256)[None, :])


def test_patchify_only_equals_full_path_at_identity_size():
    """With the target equal to the source size the resize is the identity
    (pinned above), so the full path and the patchify-only path agree
    exactly, images and odd counts included."""
    rng = np.random.default_rng(32)
    f = rng.integers(0, 256, size=(4, 96, 64, 3), dtype=np.uint8)
    mean, std = (0.3, 0.4, 0.5), (0.2, 0.25, 0.3)
    for idx in ([1, 3], [2], [0, 3, 1], [3, 3, 0, 1]):
        assert np.array_equal(oracle.patchify_item(f, idx, mean, std),
                              oracle.preprocess_item(f, idx, 96, 64, mean, std))


def test_patchify_only_constant_frame_closed_form():
    f = np.full((1, 32, 64, 3), 200, np.uint8)
    mean, std = (0.481, 0.458, 0.408), (0.269, 0.261, 0.276)
    rows = oracle.patchify_item(f, [0], mean, std)
    for c in range(3):
        assert np.all(rows[:, 512 * c:512 * (c + 1)] == (200 / 255 - mean[c]) / std[c])


def test_patchify_only_errors():
    f = np.zeros((2, 32, 48, 3), np.uint8)               # 48 is not a multiple of 32
    with pytest.raises(oracle.OracleError) as e:
        oracle.patchify_item(f, [0, 1], (0.5,) * 3, (0.5,) * 3)
    assert e.value.code == oracle.ERR_DIMS
    f = np.zeros((2, 32, 64, 3), np.uint8)
    with pytest.raises(oracle.OracleError) as e:
        oracle.patchify_item(f, [0, 2], (0.5,) * 3, (0.5,) * 3)
    assert e.value.code == oracle.ERR_INDEX


# -- uint8 cache writer (fixed-point resampling) ----------------------------

PIL_SHAPES = [
    (64, 96, 32, 48), (240, 320, 128, 160), (40, 50, 64, 96), (100, 60, 64, 96),
    (96, 128, 96, 128), (1, 1, 32, 32), (300, 20, 32, 32), (77, 131, 64, 96),
    (720, 1280, 256, 448), (480, 854, 352, 640), (723, 740, 736, 736), (333, 257, 320, 256),
]


@pytest.mark.parametrize("H,W,h,w", PIL_SHAPES)
def test_resize_u8_equals_pillow_bicubic(H, W, h, w):
    """The fixed-point cache writer reproduces Pillow's BICUBIC resize of an
    RGB image byte for byte (an independent implementation of the same
    conventions), on noise and on a smooth ramp with clipping overshoot."""
    PIL = pytest.importorskip("PIL.Image")
    rng = np.random.default_rng(H * 7919 + W)
    noise = rng.integers(0, 256, size=(H, W, 3), dtype=np.uint8)
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    ramp = np.stack([(xx * 255 // max(W - 1, 1)), (yy * 255 // max(H - 1, 1)),
                     ((xx + yy) % 2) * 255], axis=-1).astype(np.uint8)
    for img in (noise, ramp):
        ref = np.asarray(PIL.fromarray(img, "RGB").resize((w, h), PIL.BICUBIC))
        assert np.array_equal(oracle.resize_u8(img, h, w), ref)


# Float resampling at the workloads' shapes: the 240x320, 480x854, 1080x1920
# and 720x1280 videos, the three video sizes of the mixed batch, two of its
# images (one upscaled) and a small upscale.
PIL_FLOAT_SHAPES = [
    (240, 320, 128, 160), (480, 854, 352, 640), (1080, 1920, 448, 800), (720, 1280, 256, 448),
    (360, 640, 320, 576), (720, 1280, 320, 576), (333, 257, 320, 256), (1000, 712, 992, 704),
    (40, 50, 64, 96),
]


@pytest.mark.parametrize("H,W,h,w", PIL_FLOAT_SHAPES)
def test_resize_frame_equals_pillow_float_bicubic(H, W, h, w):
    """The float resampling (no rounding or clamping between passes) agrees
    with Pillow's BICUBIC resize of 32-bit float images ('F' mode), an
    independent implementation of the same antialiased Keys filter, per
    channel.  Pillow keeps its intermediate and result in float32, which
    puts its values within a few 1e-5 pixel levels of the double-precision
    ones; a wrong filter parameter, window or normalisation is off by far
    more than the 1e-4 allowed."""
    PIL = pytest.importorskip("PIL.Image")
    rng = np.random.default_rng(H * 31 + W * 7 + h)
    frame = rng.integers(0, 256, size=(H, W, 3), dtype=np.uint8)
    ours = oracle.resize_frame(frame, h, w)
    for c in range(3):
        ref = np.asarray(PIL.fromarray(frame[:, :, c].astype(np.float32), "F").resize((w, h), PIL.BICUBIC),
                         dtype=np.float64)
        assert np.abs(ours[c] - ref).max() <= 1e-4


def test_fixed_weights_are_rounded_float_weights():
    # exact 2x downscale interior: the dyadic weights scale to integers
    lo, q = oracle.fixed_weights(320, 160, 40)
    assert lo == 77
    assert q.tolist() == [round(v * 2 ** 22) for v in
                          [-0.01171875, -0.03515625, 0.11328125, 0.43359375,
                           0.43359375, 0.11328125, -0.03515625, -0.01171875]]
    # identity: one weight of exactly 2^22
    lo, q = oracle.fixed_weights(96, 96, 10)
    assert q.tolist() == [0, 1 << 22, 0, 0] and lo == 9
    # every window: within half a unit of the float weight, sums near 2^22
    for n_in, n_out in [(720, 256), (1280, 448), (40, 64), (1080, 448)]:
        for i in range(0, n_out, 7):
            lo, q = oracle.fixed_weights(n_in, n_out, i)
            lo2, wf = oracle.filter_weights(n_in, n_out, i)
            assert lo == lo2 and len(q) == len(wf)
            assert np.all(np.abs(q - wf * 2 ** 22) <= 0.5)
            assert abs(int(q.sum()) - (1 << 22)) <= len(q)


def test_resize_u8_constant_identity_and_range():
    f = np.full((50, 70, 3), 173, np.uint8)
    assert np.all(oracle.resize_u8(f, 32, 64) == 173)
    rng = np.random.default_rng(9)
    g = rng.integers(0, 256, size=(64, 96, 3), dtype=np.uint8)
    assert np.array_equal(oracle.resize_u8(g, 64, 96), g)
    # where nothing clips (a smooth frame inside [16, 239]) the only
    # difference from the real-valued resize is the rounding after each pass:
    # at most one level from the rounded real value
    yy, xx = np.meshgrid(np.arange(64), np.arange(96), indexing="ij")
    smooth = np.stack([16 + (xx * 223) // 95, 16 + (yy * 223) // 63,
                       16 + ((xx + 2 * yy) * 223) // 221], axis=-1).astype(np.uint8)
    real = oracle.resize_frame(smooth, 32, 64)                 # [3][h][w]
    ref = np.floor(real + 0.5).transpose(1, 2, 0)
    assert np.abs(oracle.resize_u8(smooth, 32, 64).astype(int) - ref).max() <= 1


def test_resize_u8_item_order_and_errors():
    rng = np.random.default_rng(10)
    f = rng.integers(0, 256, size=(4, 40, 60, 3), dtype=np.uint8)
    out = oracle.resize_u8_item(f, [3, 0, 3], 32, 64)
    assert out.shape == (3, 32, 64, 3)
    for k, src in enumerate([3, 0, 3]):
        assert np.array_equal(out[k], oracle.resize_u8(f[src], 32, 64))
    with pytest.raises(oracle.OracleError) as e:
        oracle.resize_u8_item(f, [4], 32, 64)
    assert e.value.code == oracle.ERR_INDEX
    with pytest.raises(oracle.OracleError) as e:
        oracle.resize_u8_item(f, [0], 30, 64)
    assert e.value.code == oracle.ERR_DIMS


# -- position tables ---------------------------------------------------------

def test_position_ids_read_back_from_patchified_coordinates():
    """Patchify frames whose pixels hold their own patch coordinates: each
    row's content then names its patch, which must be the row's ViT position
    (and its window's LLM position)."""
    H, W = 64, 96
    ii, jj = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    vals = np.zeros((4, 3, H, W), np.int64)
    for fr in range(4):
        vals[fr, 0] = ii // 16
        vals[fr, 1] = jj // 16
        vals[fr, 2] = 10 * (fr // 2)                     # frame pair
    f = _identity_item(vals)
    rows = oracle.patchify_item(f, [0, 1, 2, 3], (0.0,) * 3, (1 / 255,) * 3)
    vit, llm, cu = oracle.position_ids([4], [H], [W])
    got = np.stack([np.rint(rows[:, 1024]) // 10, np.rint(rows[:, 0]), np.rint(rows[:, 512])], 1)
    assert np.array_equal(vit, got.astype(np.int64))
    assert np.array_equal(llm, np.stack([vit[::4, 0], vit[::4, 1] // 2, vit[::4, 2] // 2], 1))
    assert cu.tolist() == [0, 24, 48]


def test_position_ids_by_reshape_and_ragged_segments():
    n_idx, hs, ws = [3, 1, 4], [64, 96, 32], [32, 64, 160]
    vit, llm, cu = oracle.position_ids(n_idx, hs, ws)
    parts = []
    for n, h, w in zip(n_idx, hs, ws):
        t, hm, wm = (n + 1) // 2, h // 32, w // 32
        tt, bh, bw, mh, mw = np.meshgrid(np.arange(t), np.arange(hm), np.arange(wm),
                                         np.arange(2), np.arange(2), indexing="ij")
        parts.append(np.stack([tt, 2 * bh + mh, 2 * bw + mw], -1).reshape(-1, 3))
    assert np.array_equal(vit, np.concatenate(parts))
    assert np.array_equal(llm[:, 1:], vit[::4, 1:] // 2) and np.array_equal(llm[:, 0], vit[::4, 0])
    # one segment per frame pair: 2 + 1 + 2 pairs
    assert cu.tolist() == [0, 8, 16, 40, 60, 80]
    _, ocu = oracle.layout(n_idx, hs, ws)
    assert cu[-1] == ocu[-1] == len(vit)


# -- Qwen2/2.5-VL geometry: patch 14, merge windows of 28, rows of 1176 -----

def test_smart_resize_factor_28_worked_values():
    # 720x1280 under 262,144 px: beta = sqrt(921600/262144) = 1.875,
    # floor(720/1.875/28) = 13, floor(1280/1.875/28) = 24
    assert oracle.smart_resize(720, 1280, 28, 0, 262144) == (364, 672)
    # 480x854 under 230,400 px: rhe(854/28 = 30.5) = 30 first, then the
    # budget branch: floor(12.85) = 12, floor(22.87) = 22
    assert oracle.smart_resize(480, 854, 28, 0, 230400) == (336, 616)
    assert oracle.smart_resize(1024, 1024, 28, 0, 1003520) == (980, 980)
    h, w = oracle.smart_resize(333, 257, 28, 65536, 1003520)
    assert h % 28 == 0 and w % 28 == 0


def test_patch14_inverse_by_reshape_full_and_patchify_paths():
    rng = np.random.default_rng(61)
    n, H, W = 3, 56, 84
    f = rng.integers(0, 256, size=(n, H, W, 3), dtype=np.uint8)
    mean, std = (0.48, 0.46, 0.41), (0.27, 0.26, 0.28)
    idx = [2, 0, 1]                                           # padded with 1
    ref = (f[[2, 0, 1, 1]].transpose(0, 3, 1, 2) / 255.0 - np.array(mean)[None, :, None, None]) \
        / np.array(std)[None, :, None, None]
    for rows in (oracle.patchify_item(f, idx, mean, std, patch=14),
                 oracle.preprocess_item(f, idx, H, W, mean, std, patch=14)):
        t, hm, wm = 2, H // 28, W // 28
        assert rows.shape == (t * hm * wm * 4, 1176)
        v = rows.reshape(t, hm, wm, 2, 2, 3, 2, 14, 14).transpose(0, 6, 5, 1, 3, 7, 2, 4, 8)
        np.testing.assert_allclose(v.reshape(2 * t, 3, H, W), ref, rtol=0, atol=1e-12)


def test_patch14_row_and_column_order():
    H, W = 28, 84
    vals = np.zeros((2, 3, H, W), np.int64)
    ii, jj = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    vals[:, 0] = 10 * (ii // 14) + (jj // 14)
    for fr in range(2):
        vals[fr, 1] = 50 + 10 * fr
        vals[fr, 2] = 14 * (ii % 14) + (jj % 14)
    f = _identity_item(vals)
    rows = oracle.patchify_item(f, [0, 1], (0.0,) * 3, (1 / 255,) * 3, patch=14)
    assert rows.shape == (12, 1176)
    assert np.rint(rows[:, :196].mean(1)).astype(int).tolist() == [0, 1, 10, 11, 2, 3, 12, 13, 4, 5, 14, 15]
    assert np.allclose(rows[:, 392:588], 50) and np.allclose(rows[:, 588:784], 60)
    assert np.allclose(rows[:, 784:980], np.arange(196)[None, :])


def test_patch14_layout_and_positions():
    g, cu = oracle.layout([8, 1], [364, 980], [672, 980], patch=14)
    assert g.tolist() == [[4, 26, 48], [1, 70, 70]]
    assert cu.tolist() == [0, 4 * 26 * 48, 4 * 26 * 48 + 4900]
    assert oracle.item_rows(256, 252, 448, 14) == 128 * 18 * 32
    with pytest.raises(oracle.OracleError) as e:
        oracle.layout([2], [64], [64], patch=14)              # not a multiple of 28
    assert e.value.code == oracle.ERR_DIMS
    vit, llm, vcu = oracle.position_ids([3], [56], [84], patch=14)
    t, hm, wm = 2, 2, 3
    tt, bh, bw, mh, mw = np.meshgrid(np.arange(t), np.arange(hm), np.arange(wm), np.arange(2),
                                     np.arange(2), indexing="ij")
    assert np.array_equal(vit, np.stack([tt, 2 * bh + mh, 2 * bw + mw], -1).reshape(-1, 3))
    assert vcu.tolist() == [0, 24, 48]
