"""Write tests/golden/tiny_3steps.json: the oracle's trajectory on the tiny
workload (2 detached blocks 16->32->32 + BCE heads, M=64, Adam lr 1e-3,
seed 0, 3 steps, one fresh batch per step).  Calls only the oracle and the
input generator; rerun only when the oracle's arithmetic changes for a
reason tied to the paper."""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from paper_2608_18469_amd import synth  # noqa: E402


def trajectory():
    cfg = synth.config("tiny")
    params, batches = synth.make_workload(cfg, 0, 3)
    m, v = synth.zero_state(params), synth.zero_state(params)
    p, t = params, 0
    rec = []
    for x, y in batches:
        r = oracle.step(cfg, p, m, v, t, x, y)
        p, m, v, t = r["params"], r["m"], r["v"], r["t"]
        rec.append({
            "losses": r["losses"],
            "grad_norms": [float(np.sqrt(sum(float(np.sum(np.asarray(a) ** 2)) for (W, b) in g["layers"] for a in (W, b))
                                         + sum(float(np.sum(np.asarray(a) ** 2)) for a in g["head"]))) for g in r["grads"]],
            "head_c": [float(q["head"][1][0]) for q in p],
            "W1_00": [float(q["layers"][0][0][0, 0]) for q in p],
        })
    return rec


if __name__ == "__main__":
    out = {"workload": "tiny (2 blocks 16->32->32, fp32, M=64, seed 0, 3 steps)",
           "source": "oracle/erase_oracle.py step(), float64", "steps": trajectory()}
    with open(os.path.join(HERE, "tiny_3steps.json"), "w") as f:
        json.dump(out, f, indent=1)
