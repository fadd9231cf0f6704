"""Write tests/golden/*.json from the oracle alone (run: python tests/golden/make_golden.py).

The fixtures freeze the oracle's codes, scales and accumulators on tiny seeded
layers, so that a later change to the oracle's arithmetic shows up as a diff.
Inputs come from the package's seeded generators; values come only from
``oracle/``.
"""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import backward as BW          # noqa: E402
from paper_2010_14298_amd import synth      # noqa: E402

CASES = {
    "linear_psq8": dict(n=8, d_in=12, d_out=16, qb_x=("psq", 8, 0)),
    "linear_ptq4": dict(n=8, d_in=12, d_out=16, qb_x=("ptq", 4, 0)),
    "linear_bhq5_k4": dict(n=10, d_in=12, d_out=16, qb_x=("bhq", 5, 4)),
}


def case(name):
    c = CASES[name]
    X, W, G = synth.linear_small(seed=0, n=c["n"], d_in=c["d_in"], d_out=c["d_out"])
    r = BW.linear_backward(X, W, G, qb_x=c["qb_x"], seed=0)
    out = dict(
        qx_scale=float(r["qx"]["scale"]), qx_zero=float(r["qx"]["zero"]),
        qb1_code=r["qb1"]["code"].tolist(), qb2_code=r["qb2"]["code"].tolist(),
        qb2_scale=np.atleast_1d(r["qb2"]["scale"]).astype(float).tolist(),
        qb2_zero=np.atleast_1d(r["qb2"]["zero"]).astype(float).tolist(),
        acc_w=r["acc_w"].tolist(), acc_x=r["acc_x"].tolist(),
        grad_W=r["grad_W"].astype(float).tolist(), grad_X=r["grad_X"].astype(float).tolist(),
    )
    if "perm" in r["qb2"]:
        out["perm"] = r["qb2"]["perm"].tolist()
    return out


if __name__ == "__main__":
    for name in CASES:
        with open(os.path.join(HERE, name + ".json"), "w") as f:
            json.dump(dict(case=name, spec=CASES[name], result=case(name)), f, indent=None)
        print("wrote", name)
