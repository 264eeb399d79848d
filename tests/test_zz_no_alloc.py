"""vp_preprocess_batch_noalloc (the entry point that allocates nothing: its
plan goes to the library's fixed device memory) against vp_preprocess_batch
through the C ABI: the same rows, bit for bit, with the same grid_thw and
cu_seqlens, on two calls in a row -- the second with a smaller batch, whose
plan is shorter than the one the fixed memory still holds -- in both output
types.  Rows past the batch must stay untouched.
"""
import sys

import numpy as np
import pytest

import paper_2604_16893_amd as vp
import workloads

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def log(msg):
    print(f"[no-alloc] {msg}", flush=True)
    sys.stdout.flush()


def _items(specs, seed):
    out = []
    for k, (n_src, H, W, idx, h, w) in enumerate(specs):
        it = workloads.Item("video", n_src, H, W, "uniform", seed + k, {"mode": "uniform", "n": 1})
        out.append(vp.Item(workloads.frames_torch(it, DEV), np.asarray(idx, np.int32), h, w))
    return out


# a ragged batch of five kernel shapes (several launches), then a smaller one
FIRST = [(9, 120, 200, [0, 3, 8, 5], 96, 160), (1, 333, 257, [0], 320, 256),
         (7, 45, 80, [6], 64, 64), (3, 480, 854, [0, 1, 2], 128, 224),
         (2, 300, 3000, [1, 0], 32, 96), (4, 720, 1280, [3, 1, 0, 2], 256, 448)]
SECOND = [(3, 75, 101, [2, 0, 1], 64, 96), (1, 250, 333, [0], 256, 320)]


def _run_both(items, dtype):
    mean, std = (0.481, 0.458, 0.408), (0.269, 0.261, 0.276)
    code = vp.VP_OUT_BF16 if dtype == "bf16" else vp.VP_OUT_F32
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    grid, cu, rows, ws = vp.vp_batch_layout(items)
    assert ws <= vp.VP_NOALLOC_PLAN_BYTES
    ref = torch.full((rows + 4, 1536), float("nan"), dtype=tdt, device=DEV)
    work = torch.empty(ws, dtype=torch.uint8, device=DEV)
    g1, c1 = vp.vp_preprocess_batch(items, mean, std, code, ref, work)
    got = torch.full((rows + 4, 1536), float("nan"), dtype=tdt, device=DEV)
    g2, c2 = vp.vp_preprocess_batch_noalloc(items, mean, std, code, got)
    torch.cuda.synchronize()
    assert g1.tolist() == g2.tolist() == grid.tolist()
    assert c1.tolist() == c2.tolist() == cu.tolist()
    assert torch.isnan(got[rows:].float()).all(), "rows past the batch were written"
    a = got[:rows].view(torch.int16 if dtype == "bf16" else torch.int32)
    b = ref[:rows].view(torch.int16 if dtype == "bf16" else torch.int32)
    same = torch.equal(a, b)
    log(f"{len(items)} items, {rows} rows, plan {ws} bytes, {dtype}: bit-identical {same}")
    assert same


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_workspace_entry_twice(dtype):
    first = _items(FIRST, 300)
    second = _items(SECOND, 400)
    assert vp.vp_batch_layout(second)[3] < vp.vp_batch_layout(first)[3]
    _run_both(first, dtype)
    _run_both(second, dtype)


def test_noalloc_on_a_side_stream_in_order():
    """Two calls on one non-default stream are ordered: the second (smaller)
    call's plan copy waits for the first call's kernels."""
    first = _items(FIRST, 500)
    second = _items(SECOND, 600)
    mean, std = (0.5, 0.5, 0.5), (0.5, 0.5, 0.5)
    outs = []
    s = torch.cuda.Stream()
    for items in (first, second):
        _, _, rows, _ = vp.vp_batch_layout(items)
        outs.append(torch.full((rows, 1536), float("nan"), dtype=torch.bfloat16, device=DEV))
    with torch.cuda.stream(s):
        vp.vp_preprocess_batch_noalloc(first, mean, std, vp.VP_OUT_BF16, outs[0], s)
        vp.vp_preprocess_batch_noalloc(second, mean, std, vp.VP_OUT_BF16, outs[1], s)
    torch.cuda.synchronize()
    for items, got in zip((first, second), outs):
        ref, _, _ = vp.preprocess(items, mean, std, "bf16")
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.int16), ref.view(torch.int16))
