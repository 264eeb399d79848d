"""GPU parity of the normalise+patchify-only entry (vp_patchify_batch).

Frames already at the target size are normalised and patchified through the
C ABI and compared with the oracle's patchify-only definition: element by
element on small cases (float32 within 2e-5, bfloat16 within one ulp or
2e-5), bit for bit against vp_preprocess_batch at identity size (the same
arithmetic), and on whole sampled frame pairs of the full-size cached
counterpart of the 64 x 256-frame workload.  A NaN sentinel proves every
output row was written and none beyond.
"""
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
    print(f"[gpu-patchify] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _free_memory():
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def run(entry, items, mean, std, dtype, extra_rows=8, patch=16):
    """items: list of (device frames, indices); every target is its frames' size."""
    vitems = [vp.Item(f, idx, f.shape[1], f.shape[2], patch) for f, idx in items]
    grid, cu, rows, ws = vp.vp_batch_layout(vitems)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = torch.full((rows + extra_rows, vp.row_width(patch)), float("nan"), dtype=tdt, device=DEV)
    work = torch.empty(ws, dtype=torch.uint8, device=DEV)
    g2, cu2 = entry(vitems, mean, std, vp.VP_OUT_BF16 if dtype == "bf16" else vp.VP_OUT_F32,
                    out, work)
    torch.cuda.synchronize()
    assert g2.tolist() == grid.tolist() and cu2.tolist() == cu.tolist()
    og, ocu = oracle.layout([len(i[1]) for i in items], [i[0].shape[1] for i in items],
                            [i[0].shape[2] for i in items], patch=patch)
    assert grid.tolist() == og.tolist() and cu.tolist() == ocu.tolist()
    if extra_rows:
        assert torch.isnan(out[rows:].float()).all(), "rows beyond the batch were written"
    assert not torch.isnan(out[:rows].float()).any(), "a row of the batch was not written"
    return out[:rows], cu


def host_rows(out, lo, hi, dtype):
    t = out[lo:hi]
    if dtype == "bf16":
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def assert_close(gpu, ref, dtype, what):
    res = compare.check_bf16(gpu, ref) if dtype == "bf16" else compare.check_f32(gpu, ref)
    log(f"{what}: {res}")
    assert res["ok"], f"{what}: {res}"


def _frames(seed, n, h, w):
    it = workloads.Item("video", n, h, w, "uniform", seed, {"mode": "uniform", "n": n})
    return workloads.frames_torch(it, DEV), workloads.frames_np(it)


MEAN, STD = (0.481, 0.458, 0.408), (0.269, 0.261, 0.276)

CASES = [
    # name, [(n_src, h, w, indices)], dtype
    ("one_window", [(2, 32, 32, [0, 1])], "f32"),
    ("video_reordered", [(5, 64, 96, [4, 0, 2, 1])], "f32"),
    ("odd_count_bf16", [(3, 96, 64, [2, 0, 1])], "bf16"),
    ("image", [(1, 256, 320, [0])], "bf16"),
    ("wide_row", [(2, 32, 1024, [1, 0])], "f32"),
    ("ragged_batch", [(4, 64, 64, [3, 1]), (1, 128, 96, [0]), (6, 32, 160, [5, 5, 0, 2, 4]),
                      (2, 224, 32, [1, 0])], "bf16"),
]


@pytest.mark.parametrize("name,specs,dtype", CASES, ids=[c[0] for c in CASES])
def test_patchify_small_cases_vs_oracle(name, specs, dtype):
    items, host = [], []
    for k, (n, h, w, idx) in enumerate(specs):
        fd, fh = _frames(200 + k, n, h, w)
        items.append((fd, np.asarray(idx, np.int32)))
        host.append(fh)
    log(f"case {name}: {[(s[0], s[1], s[2]) for s in specs]} {dtype}")
    out, cu = run(vp.vp_patchify_batch, items, MEAN, STD, dtype)
    for k, (fd, idx) in enumerate(items):
        ref = oracle.patchify_item(host[k], idx, MEAN, STD)
        assert_close(host_rows(out, cu[k], cu[k + 1], dtype), ref, dtype, f"{name} item {k}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_patchify_equals_preprocess_at_identity_size(dtype):
    """Same bytes, same arithmetic: the identity resize of vp_preprocess_batch
    and vp_patchify_batch agree bit for bit."""
    items = []
    for k, (n, h, w, idx) in enumerate([(4, 64, 96, [3, 0, 1]), (1, 96, 128, [0])]):
        fd, _ = _frames(300 + k, n, h, w)
        items.append((fd, np.asarray(idx, np.int32)))
    log(f"identity vs patchify {dtype}")
    a, _ = run(vp.vp_patchify_batch, items, MEAN, STD, dtype)
    b, _ = run(vp.vp_preprocess_batch, items, MEAN, STD, dtype)
    assert torch.equal(a.view(torch.int16) if dtype == "bf16" else a.view(torch.int32),
                       b.view(torch.int16) if dtype == "bf16" else b.view(torch.int32))


def test_patchify_cached_workload_full_size():
    """The cached counterpart of the 64 x 256-frame workload at full size:
    every row written, and whole frame pairs of several items against the
    oracle."""
    wl = workloads.patchify_config()
    log(f"workload {wl.name}")
    items = []
    for it in wl.items:
        idx = vp.vp_sample_indices(it.n_src, vp.VP_SAMPLE_UNIFORM, it.sample["n"])
        items.append((workloads.frames_torch(it, DEV, chunk=64), idx))
    out, cu = run(vp.vp_patchify_batch, items, wl.mean, wl.std, wl.out_dtype, extra_rows=4)
    rng = np.random.default_rng(41)
    per_pair = (256 // 16) * (448 // 16)
    for k in rng.choice(len(items), size=4, replace=False):
        it = wl.items[int(k)]
        idx = items[int(k)][1]
        tt = int(rng.integers(0, len(idx) // 2))
        pair = idx[2 * tt:2 * tt + 2]
        ref = oracle.patchify_item(workloads.frames_np(it, pair), [0, 1], wl.mean, wl.std)
        lo = int(cu[k]) + tt * per_pair
        assert_close(host_rows(out, lo, lo + per_pair, wl.out_dtype), ref, wl.out_dtype,
                     f"cached workload item {int(k)} pair {tt}")


CASES14 = [
    ("p14_one_window", [(2, 28, 28, [0, 1])], "f32"),
    ("p14_video", [(5, 56, 84, [4, 0, 2, 1])], "bf16"),
    ("p14_odd_and_image", [(3, 84, 56, [2, 0, 1]), (1, 252, 448, [0])], "bf16"),
    ("p14_wide_rows", [(2, 28, 1008, [1, 0])], "f32"),
]


@pytest.mark.parametrize("name,specs,dtype", CASES14, ids=[c[0] for c in CASES14])
def test_patchify_patch14_vs_oracle(name, specs, dtype):
    items, host = [], []
    for k, (n, h, w, idx) in enumerate(specs):
        fd, fh = _frames(700 + k, n, h, w)
        items.append((fd, np.asarray(idx, np.int32)))
        host.append(fh)
    log(f"case {name}: {[(s[0], s[1], s[2]) for s in specs]} {dtype}")
    out, cu = run(vp.vp_patchify_batch, items, MEAN, STD, dtype, patch=14)
    for k, (fd, idx) in enumerate(items):
        ref = oracle.patchify_item(host[k], idx, MEAN, STD, patch=14)
        assert_close(host_rows(out, cu[k], cu[k + 1], dtype), ref, dtype, f"{name} item {k}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_patch14_patchify_equals_preprocess_at_identity_size(dtype):
    items = []
    for k, (n, h, w, idx) in enumerate([(4, 56, 84, [3, 0, 1]), (1, 112, 56, [0])]):
        fd, _ = _frames(800 + k, n, h, w)
        items.append((fd, np.asarray(idx, np.int32)))
    a, _ = run(vp.vp_patchify_batch, items, MEAN, STD, dtype, patch=14)
    b, _ = run(vp.vp_preprocess_batch, items, MEAN, STD, dtype, patch=14)
    assert torch.equal(a.view(torch.int16) if dtype == "bf16" else a.view(torch.int32),
                       b.view(torch.int16) if dtype == "bf16" else b.view(torch.int32))

