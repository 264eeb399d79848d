"""GPU parity of the position tables (vp_position_ids): the ViT row
coordinates, the LLM window coordinates and the ViT segments, bit-exact
against the oracle on a ragged batch and at full size for the 64 x 256-frame
workload (3,670,016 rows), with sentinels proving that nothing past the
batch was written."""
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
    print(f"[gpu-positions] {msg}", flush=True)
    sys.stdout.flush()


def _check(items_spec, patch=16):
    # frames are never read: any valid device pointer will do
    dummy = torch.zeros((1, 32, 32, 3), dtype=torch.uint8, device=DEV)
    items = [vp.Item((dummy.data_ptr(), n_src, 32, 32), idx, h, w, patch)
             for n_src, idx, h, w in items_spec]
    _, _, rows, ws = vp.vp_batch_layout(items)
    vit = torch.full((rows + 4, 3), -7, dtype=torch.int32, device=DEV)
    llm = torch.full((rows // 4 + 2, 3), -7, dtype=torch.int32, device=DEV)
    work = torch.empty(ws, dtype=torch.uint8, device=DEV)
    cu = vp.vp_position_ids(items, vit, llm, work)
    torch.cuda.synchronize()
    ov, ol, ocu = oracle.position_ids([len(s[1]) for s in items_spec], [s[2] for s in items_spec],
                                      [s[3] for s in items_spec], patch=patch)
    v = vit.cpu().numpy()
    l = llm.cpu().numpy()
    assert np.array_equal(v[:rows], ov) and (v[rows:] == -7).all()
    assert np.array_equal(l[:rows // 4], ol) and (l[rows // 4:] == -7).all()
    assert cu.tolist() == ocu.tolist()
    log(f"{len(items_spec)} items, {rows} rows, {len(cu) - 1} segments: equal")


def test_positions_ragged_batch():
    _check([(5, [4, 0, 2], 64, 32), (1, [0], 96, 64), (9, [0, 3, 8, 5], 96, 160),
            (3, [1, 2, 0, 1, 2], 320, 576), (1, [0], 992, 992)])


def test_positions_rollout_workload_full_size():
    wl = workloads.config(4)
    _check([(it.n_src, list(range(256)), 256, 448) for it in wl.items])


def test_positions_patch14_ragged_batch():
    _check([(5, [4, 0, 2], 56, 28), (1, [0], 84, 56), (3, [1, 2, 0, 1, 2], 252, 448),
            (1, [0], 980, 980)], patch=14)

