"""Writes exact_regime.json: small integer-valued inputs and the oracle's
results for them (run from the repository root:
``python -m tests.golden.make_golden``).

In this regime (integers of magnitude <= 64, K <= 8, eta = 1/8, rho = 1/2)
every intermediate of the reduction (Sec. 3.2, Sec. 5) and of the elastic
step (Sec. 2.1 Eq. 1, Sec. 2.2 Eqs. 2-3) is exactly representable in
binary32, so any correct implementation returns these exact bits whatever
its order of operations.  The script calls only the oracle.
"""

import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
import oracle  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "exact_regime.json")


def main():
    orc = oracle.load()
    rng = np.random.default_rng(20180111)
    N = 37  # not a multiple of 4: exercises a ragged tail
    cases = {"reduce": [], "easgd": []}
    for K in (1, 2, 3, 4, 8):
        ins = [rng.integers(-64, 65, N).astype(np.float32) for _ in range(K)]
        case = {"K": K, "in": [a.tolist() for a in ins], "sum": orc.reduce(ins, oracle.SUM).tolist()}
        if K & (K - 1) == 0:  # power of two: the average is exact too
            case["avg"] = orc.reduce(ins, oracle.AVG).tolist()
        cases["reduce"].append(case)
    eta, rho = 0.125, 0.5
    for K in (1, 3, 4, 8):
        xs = [rng.integers(-64, 65, N).astype(np.float32) for _ in range(K)]
        gs = [rng.integers(-64, 65, N).astype(np.float32) for _ in range(K)]
        xc = rng.integers(-64, 65, N).astype(np.float32)
        x64 = [a.astype(np.float64) for a in xs]
        c64 = xc.astype(np.float64)
        orc.easgd_step(x64, gs, c64, eta, rho)
        for a in x64 + [c64]:
            assert np.array_equal(a.astype(np.float32).astype(np.float64), a)
        cases["easgd"].append({"K": K, "eta": eta, "rho": rho,
                               "x": [a.tolist() for a in xs], "g": [a.tolist() for a in gs],
                               "xc": xc.tolist(),
                               "x_out": [a.tolist() for a in x64], "xc_out": c64.tolist()})
    with open(OUT, "w") as f:
        json.dump({"about": "integer-valued inputs whose results are exact in binary32; "
                            "written by tests/golden/make_golden.py from the CPU oracle",
                   "N": N, **cases}, f, separators=(",", ":"))


if __name__ == "__main__":
    main()
