"""Write tests/golden/oracle_tiny.json: oracle outputs for one tiny seeded case.

Calls only the oracle and the seeded input generators.  The fixture guards the
oracle against unnoticed drift: any later change to its arithmetic must come
with a regenerated fixture and a commit message that names the passage of the
paper (FlowTT) justifying it.
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
import ttgen  # noqa: E402

CASE = dict(seed=2026, T=2, n=(3, 4, 5), d=(2, 2, 2), R=3, B=4, max_len=4)


def make_case():
    return ttgen.tiny(CASE["seed"], CASE["T"], CASE["n"], CASE["d"], CASE["R"], B=CASE["B"],
                      max_len=CASE["max_len"])


def main():
    oracle.build(force=False)
    case = make_case()
    V, _ = oracle.forward(case)
    dG1, dG2, dG3, _ = oracle.backward(case)
    grp = oracle.grouping(case)
    out = dict(case=CASE, V=[repr(float(x)) for x in V.ravel()],
               dG1=[repr(float(x)) for x in dG1.ravel()], dG2=[repr(float(x)) for x in dG2.ravel()],
               dG3=[repr(float(x)) for x in dG3.ravel()],
               uniq_g=[int(x) for x in grp["uniq_g"]], pg_q=[int(x) for x in grp["pg_q"]])
    with open(os.path.join(HERE, "oracle_tiny.json"), "w") as f:
        json.dump(out, f, indent=0)


if __name__ == "__main__":
    main()
