"""Oracle against the hand-derived fixtures in tests/golden/.

The paper prints no worked numerical example, so the fixtures are small
cases derived by hand from the lattice definitions; each file states its
derivation.
"""
import math
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _num(tok):
    return float(eval(tok, {"__builtins__": {}}, {"sqrt": math.sqrt, "pi": math.pi}))


def load_simplex_cases():
    cases, cur = [], None
    with open(os.path.join(GOLDEN, "simplex_hand.txt")) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            tok = line.split()
            if tok[0] == "case":
                cur = {"name": tok[1], "d": int(tok[3]), "keys": {}}
                cases.append(cur)
            elif tok[0] == "p":
                cur["p"] = [_num(t) for t in tok[1:]]
            elif tok[0] == "key":
                cur["keys"][int(tok[1])] = [int(t) for t in tok[2:]]
            elif tok[0] == "bary":
                cur["bary"] = [_num(t) for t in tok[1:]]
            elif tok[0] == "rank":
                cur["rank"] = [int(t) for t in tok[1:]]
    return cases


@pytest.mark.parametrize("case", load_simplex_cases(), ids=lambda c: c["name"])
def test_hand_derived_simplex(O, case):
    d = case["d"]
    s = O.simplex(np.array([case["p"]], dtype=np.float32))
    for k in range(d + 1):
        assert s.keys[0, k].tolist() == case["keys"][k]
    np.testing.assert_allclose(s.bary[0], case["bary"], atol=2e-7)
    assert s.rank[0].tolist() == case["rank"]


def test_hand_derived_single_point_d1(O):
    vals = {}
    with open(os.path.join(GOLDEN, "single_point_d1.txt")) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                tok = line.split()
                vals[tok[0]] = tok[1:]
    p = np.array([[_num(vals["p"][0])]], dtype=np.float32)
    v = np.array([[_num(t) for t in vals["v"]]])
    gain = _num(vals["raw_gain"][0]) / _num(vals["G"][0])
    lat = O.lattice(p)
    out, _ = O.forward(lat, v, False)
    np.testing.assert_allclose(out, gain * v, rtol=1e-6)
    outn, _ = O.forward(lat, v, True)
    np.testing.assert_allclose(outn, v, rtol=1e-12)
