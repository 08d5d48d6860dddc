"""Write tests/golden/oracle_rope_causal_tiny.json: the fp64 oracle's outputs on
the tiny parity workload (B=1, H=H_kv=2, S=128, D=64, interleaved RoPE with
theta = 10000, causal mask, scale 1/8, seed 0; inputs from the seeded
generators), forward and backward, at sampled rows.

The paper prints no numeric worked example (its tables are timings), so no
stored value here is the paper's: this fixture is a regression record of the
oracle itself, written by this script, which calls only ``oracle`` and the
input generators.  ``tests/test_golden.py`` recomputes it; a change to the
oracle's arithmetic shows up as a difference against this file and has to be
justified by the passage it follows.

Run from the repository root:  python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle                                   # noqa: E402
from paper_2609_13612_amd import inputs         # noqa: E402

CASE = dict(B=1, H=2, Hkv=2, S=128, D=64, rope="interleaved", theta=10000.0, mask="causal", scale=0.125, seed=0)
ROWS = [0, 1, 2, 63, 64, 126, 127]
PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_rope_causal_tiny.json")


def compute():
    c = CASE
    t = inputs.make_qkv(c["B"], c["H"], c["Hkv"], c["S"], c["D"], seed=c["seed"], with_do=True)
    q, k, v, do = (inputs.to_f64(t[n]) for n in ("q", "k", "v", "do"))
    kw = dict(rope=c["rope"], theta=c["theta"], mask=c["mask"], scale=c["scale"])
    O, L = oracle.attention_forward(q, k, v, **kw)
    dQ, dK, dV = oracle.attention_backward(q, k, v, do, **kw)
    return {"O": O, "LSE": L, "dQ": dQ, "dK": dK, "dV": dV}


def record(res):
    out = {"case": CASE, "rows": ROWS,
           "LSE": res["LSE"][0].tolist()}
    for name in ("O", "dQ", "dK", "dV"):
        out[name] = res[name][0][:, ROWS, :].tolist()   # [head][row][dim]
    return out


if __name__ == "__main__":
    with open(PATH, "w") as f:
        json.dump(record(compute()), f)
        f.write("\n")
    print("wrote", PATH)
