"""The oracle still reproduces the committed plan fixture (a regression
anchor: a change to the oracle's sampling, smart_resize or layout arithmetic
shows up here and must be justified by the paper)."""
import json
import os

import oracle
import workloads

HERE = os.path.dirname(os.path.abspath(__file__))


def test_oracle_reproduces_plan_fixture():
    gold = json.load(open(os.path.join(HERE, "golden", "plan_configs.json")))["configs"]
    assert len(gold) == 5
    for k, g in enumerate(gold):
        wl = workloads.config(k)
        assert len(wl.items) == len(g["items"])
        for it, gi in zip(wl.items, g["items"]):
            assert (it.n_src, it.H, it.W) == (gi["n_src"], gi["H"], gi["W"])
            if it.dims is None:
                assert oracle.smart_resize(it.H, it.W, 32, it.min_pixels, it.max_pixels) == \
                    (gi["h"], gi["w"])
            s = it.sample
            if s["mode"] == "uniform":
                idx = oracle.sample_uniform(it.n_src, s["n"])
            else:
                idx = oracle.sample_fps(it.n_src, s["video_fps"], s["fps"], s["min_frames"],
                                        s["max_frames"])
            assert idx.tolist() == gi["indices"]
        grid, cu = oracle.layout([len(i["indices"]) for i in g["items"]],
                                 [i["h"] for i in g["items"]], [i["w"] for i in g["items"]])
        assert grid.tolist() == g["grid_thw"] and cu.tolist() == g["cu_seqlens"]
    # the row totals of the fixed-size workloads
    assert [g["cu_seqlens"][-1] for g in gold[:3]] == [320, 28160, 89600]
    assert gold[4]["cu_seqlens"][-1] == 3_670_016
