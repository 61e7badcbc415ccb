"""Host logic of the timing suite: Table 3's weighted ResNet-101 summary.

The summary weighs each layer's workspace by its ResNet-101 count; fed the
library's own workspace sizes at batch 1 in fp32 it must reproduce Table 3's
memory columns (sums 203.6 MB for im2col and 64.6 MB for MEC, ratio 3.2, the
paper's MB read as MiB). Timings here are made up: only the arithmetic of the
weighting is under test, no kernel runs.
"""
import json
import os

import pytest

import paper_1706_06873_amd as mec
from paper_1706_06873_amd import suite
from paper_1706_06873_amd import workloads as wl
from conftest import REPO

GOLDEN = os.path.join(REPO, "tests", "golden", "table3_resnet101_mem.json")


def fake_rows(batch=1):
    rows = []
    for i, name in enumerate(wl.TABLE3_WEIGHTS):
        layer = wl.table2_layer(name, batch)
        rows.append({"layer": layer.name, "dtype": "f32",
                     "workspace_mec": mec.workspace_bytes(*layer.dims, dtype=mec.F32),
                     "workspace_im2col": mec.im2col_bytes(*layer.dims, dtype=mec.F32),
                     "timings": {"im2col": {"us": 10.0 + i}, "lowered": {"us": 4.0 + i},
                                 "fused": {"us": 2.0 + i}}})
    return rows


def test_weights_match_table3():
    gold = json.load(open(GOLDEN))
    assert wl.TABLE3_WEIGHTS == {r["name"]: r["weight"] for r in gold["rows"]}


def test_weighted_workspace_reproduces_table3_sums():
    gold = json.load(open(GOLDEN))
    s = suite.weighted_summary(fake_rows(), 1)
    assert s["workspace_im2col_mib"] == pytest.approx(gold["sum"]["conv_mem"], abs=0.1)
    assert s["workspace_mec_mib"] == pytest.approx(gold["sum"]["mec_mem"], abs=0.1)
    assert round(s["workspace_ratio"], 1) == gold["ratio"]["conv_mem"]


def test_weighted_times():
    s = suite.weighted_summary(fake_rows(), 1)
    w = list(wl.TABLE3_WEIGHTS.values())
    assert s["im2col_us"] == pytest.approx(sum(wi * (10.0 + i) for i, wi in enumerate(w)))
    assert s["mec_fused_us"] == pytest.approx(sum(wi * (2.0 + i) for i, wi in enumerate(w)))
    assert s["time_ratio_lowered"] == pytest.approx(s["im2col_us"] / s["mec_lowered_us"], rel=1e-3)


def test_auto_sets_span_the_last_level_cache():
    """Buffer sets of the suite: a rotation through them spans at least 1 GiB
    (I, K and O of the fused form), between 2 and the cap."""
    import torch
    for name in wl.TABLE2:
        layer = wl.table2_layer(name, 32)
        I0, K0 = wl.make_inputs(layer) if name in ("cv11", "cv12") else (
            torch.empty(layer.i_n * layer.i_h * layer.i_w * layer.i_c),
            torch.empty(layer.k_h * layer.k_w * layer.i_c * layer.k_c))
        o_h, o_w = mec.output_dims(*layer.dims[1:3], *layer.dims[4:6], *layer.dims[7:9])
        o_elems = layer.i_n * o_h * o_w * layer.k_c
        sets = suite._auto_sets(I0, K0, o_elems)
        foot = I0.numel() * I0.element_size() + K0.numel() * K0.element_size() + 4 * o_elems
        assert 2 <= sets <= suite.MAX_SETS
        assert sets * foot >= suite.MIN_ROTATION_BYTES or sets == suite.MAX_SETS
        assert sets == 2 or (sets - 1) * foot < suite.MIN_ROTATION_BYTES


def test_read_sets_span_twice_the_last_level_cache():
    """Sets of an operand a kernel reads: a rotation through them spans at
    least 512 MB (twice the 256 MB last-level cache), and one set fewer would
    not, between 2 and the cap (vgg_first's 9.8 MB input: 55 sets)."""
    assert suite.READ_ROTATION_BYTES >= 2 * 256 * 10 ** 6
    for nbytes in [1, 196, 3_211_264, 9_806_208, 19_267_584, 79_149_312, 211_312_640, 2_190_000_000]:
        n = suite._read_sets(nbytes)
        assert 2 <= n <= suite.MAX_SETS
        assert n * nbytes >= suite.READ_ROTATION_BYTES or n == suite.MAX_SETS
        assert n == 2 or (n - 1) * nbytes < suite.READ_ROTATION_BYTES
    assert suite._read_sets(16 * 226 * 226 * 3 * 4) == 55


def test_bench_rotation_sets():
    """The benchmark's sets per read operand: a rotation spans at least
    512 MB (twice the 256 MB last-level cache), never fewer than asked for,
    at most 256 (vgg_first's 9.8 MB input: 55 sets; alexnet_conv1's 211 MB
    lowered tensor: 4 at the default of 4)."""
    import bench
    assert bench.READ_ROTATION_BYTES >= 2 * 256 * 10 ** 6
    assert bench.rotation_sets(16 * 226 * 226 * 3 * 4, 4) == 55
    assert bench.rotation_sets(210_946_560, 4) == 4
    assert bench.rotation_sets(210_946_560, 1) == 3
    assert bench.rotation_sets(196, 4) == 256
    for nbytes in [1, 3_211_264, 29_159_424, 79_149_312, 2_190_000_000]:
        n = bench.rotation_sets(nbytes, 1)
        assert n * nbytes >= bench.READ_ROTATION_BYTES or n == 256
        assert n == 1 or (n - 1) * nbytes < bench.READ_ROTATION_BYTES
