"""Stored hand-worked values (``tests/golden/``), each fixture citing the
passages its values follow.  The oracle and the library's planner must both
reproduce them.  No GPU."""
import json
import os

import pytest

from oracle import predictor as orc
from paper_2606_05933_amd import ssa

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _cases(name):
    with open(os.path.join(GOLDEN, name)) as f:
        data = json.load(f)
    assert data["citation"]
    return data["cases"]


@pytest.mark.parametrize("case", _cases("tab1_features_by_hand.json"))
def test_features_and_scene_by_hand(case):
    c, u = case["q_len"], case["ctx_len"]
    assert [float(v) for v in orc.features(c, u)] == [float(v) for v in case["x"]]
    assert orc.scene(c, u) == case["scene"]
    pages = max((a + b + 15) // 16 for a, b in zip(c, u))
    shape = ssa.make_shape(32, 8, 128, 1 << 16, max(pages, 1), 128 ** -0.5)
    _, info = ssa.ssa_plan(shape, c, u)
    assert [float(v) for v in info.x] == [float(v) for v in case["x"]]
    assert info.scene == case["scene"]
