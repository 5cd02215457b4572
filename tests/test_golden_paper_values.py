"""Values the paper prints, stored under tests/golden/ with their citations, against the input
recipe of the workloads and the host-side estimate the benchmark reports."""
import json
import math
import os

import pytest

from paper_2607_02829_amd import inputs
from paper_2607_02829_amd.trunk import eq_speedup_estimate

pytestmark = pytest.mark.cpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_token_counts_and_selected_tokens():
    g = _load("paper_token_counts.json")
    r = g["keep_ratio"]
    by_L = {}
    for s in g["settings"]:
        if "grid" in s:
            lat, lon = s["grid"]
            assert (lat // s["patch"]) * (lon // s["patch"]) == s["L"], s
        # K = floor(r L) reproduces the printed K of every setting
        assert math.floor(s["L"] * r) == s["K"], s
        by_L[s["L"]] = s["K"]
    # the workloads that stand in for these grids have the printed token counts and K
    for name, L in (("c1406", 8192), ("d025", 16200), ("gen", 8192), ("edm", 8192)):
        w = inputs.WORKLOADS[name]
        assert (w.L, w.keep) == (L, r), name
        assert w.K == by_L[L], name
    d025 = inputs.WORKLOADS["d025"]
    assert (d025.Hg, d025.Wg) == (720 // 8, 1440 // 8)
    assert inputs.WORKLOADS["c1406"].Hg * 2 == 128 and inputs.WORKLOADS["c1406"].Wg * 2 == 256


def test_speedup_estimate_matches_the_printed_value():
    g = _load("paper_speedup_estimate.json")
    split, r = tuple(g["split"]), g["keep_ratio"]
    est = eq_speedup_estimate(split, r)
    assert sum(split) == g["blocks"]
    assert split[0] + split[1] * r * r + split[2] == g["denominator"]
    assert est == g["blocks"] / g["denominator"]
    assert round(est, g["printed_decimals"]) == g["speedup_printed"]
    # the estimate is 1 with no routing and grows as r shrinks
    assert eq_speedup_estimate(split, 1.0) == 1.0
    assert eq_speedup_estimate(split, 0.1) > est > eq_speedup_estimate(split, 0.5)


@pytest.mark.parametrize("split,keep", [((2, 8, 2), 0.0), ((2, 8, 2), 1.5), ((-1, 8, 2), 0.25), ((0, 0, 0), 0.25)])
def test_speedup_estimate_rejects_bad_arguments(split, keep):
    with pytest.raises(ValueError):
        eq_speedup_estimate(split, keep)
