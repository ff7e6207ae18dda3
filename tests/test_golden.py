"""Oracle against the hand-derived fixtures in tests/golden/closed_forms.json."""
import json
import os

import numpy as np

from oracle import ops

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "closed_forms.json")))


def test_trilinear_axis_fixtures():
    for key in ("trilinear_axis_2_to_4", "trilinear_axis_3_to_6"):
        g = GOLD[key]
        x = np.array(g["input"])[None, None, None, None, :]
        y = ops.trilinear_fwd(x, (1, 1, len(g["output"])))
        np.testing.assert_allclose(y[0, 0, 0, 0], g["output"], atol=1e-15)


def test_ce_fixture():
    loss, _ = ops.ce_fwd_bwd(np.zeros((3, 2)), np.array([0, 1, 0]))
    assert abs(loss - GOLD["ce_uniform_two_class"]["loss"]) < 1e-15


def test_conv_all_ones_fixture():
    g = GOLD["conv_all_ones_3cube"]
    y = ops.conv3d_fwd(np.ones((1, 1, 3, 3, 3)), np.ones((1, 1, 3, 3, 3)), None, 1, 1)[0, 0]
    assert (y[1, 1, 1], y[0, 1, 1], y[0, 0, 1], y[0, 0, 0]) == (
        g["centre"], g["face"], g["edge"], g["corner"])


def test_size_chain_fixture():
    g = GOLD["size_chain_96x112x96"]
    sp = [ops.out_size(v, 7, 2, 3) for v in (96, 112, 96)]
    assert sp == g["stem"]
    for expect in g["pools"]:
        sp = [ops.out_size(v, 3, 2, 1) for v in sp]
        assert sp == expect
