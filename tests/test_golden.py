"""The exact-regime fixture (tests/golden/exact_regime.json) against the
current oracle: a change to the oracle's arithmetic that moves any of these
exact results shows up here."""

import json
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "exact_regime.json")


def test_golden_reproduced_by_oracle(orc):
    data = json.load(open(GOLDEN))
    for case in data["reduce"]:
        ins = [np.array(a, dtype=np.float32) for a in case["in"]]
        assert np.array_equal(orc.reduce(ins, oracle.SUM), np.array(case["sum"]))
        if "avg" in case:
            assert np.array_equal(orc.reduce(ins, oracle.AVG), np.array(case["avg"]))
    for case in data["easgd"]:
        xs = [np.array(a, dtype=np.float64) for a in case["x"]]
        gs = [np.array(a, dtype=np.float32) for a in case["g"]]
        xc = np.array(case["xc"], dtype=np.float64)
        orc.easgd_step(xs, gs, xc, case["eta"], case["rho"])
        for a, b in zip(xs, case["x_out"]):
            assert np.array_equal(a, np.array(b))
        assert np.array_equal(xc, np.array(case["xc_out"]))


def test_golden_values_are_integers_or_dyadic():
    """Sanity of the fixture: inputs are integers, outputs multiples of 1/16."""
    data = json.load(open(GOLDEN))
    for case in data["easgd"]:
        for a in case["x"] + case["g"] + [case["xc"]]:
            assert np.all(np.array(a) == np.round(np.array(a)))
        for a in case["x_out"] + [case["xc_out"]]:
            v = np.array(a) * 16
            assert np.all(v == np.round(v))
