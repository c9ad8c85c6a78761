"""The oracle still reproduces its committed tiny fixture (drift guard)."""
import json
import os

import numpy as np

from tests.golden.make_golden import make_case

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_oracle_matches_fixture(orc):
    ref = json.load(open(os.path.join(HERE, "oracle_tiny.json")))
    case = make_case()
    V, _ = orc.forward(case)
    dG1, dG2, dG3, _ = orc.backward(case)
    for got, key in ((V, "V"), (dG1, "dG1"), (dG2, "dG2"), (dG3, "dG3")):
        exp = np.array([float(x) for x in ref[key]])
        np.testing.assert_allclose(got.ravel(), exp, rtol=1e-13, atol=1e-15)
    grp = orc.grouping(case)
    assert grp["uniq_g"].tolist() == ref["uniq_g"]
    assert grp["pg_q"].tolist() == ref["pg_q"]
