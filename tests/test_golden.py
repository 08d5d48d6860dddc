"""The oracle against its stored regression record (tests/golden/), and that
record against closed forms.

The paper prints no numeric worked example, so the stored values are the
oracle's own, written by tests/golden/make_golden.py (oracle and input
generators only).  Two closed forms pin the record independently of the
oracle: under a causal mask row 0 attends only to key 0, so O_0 = v_0 and
LSE_0 = scale * q_0 . k_0 (RoPE is the identity at position 0).
"""
import importlib.util
import json
import os

import numpy as np

from paper_2609_13612_amd import inputs

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = os.path.join(HERE, "golden")


def _maker():
    spec = importlib.util.spec_from_file_location("make_golden", os.path.join(GOLDEN, "make_golden.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _stored():
    with open(os.path.join(GOLDEN, "oracle_rope_causal_tiny.json")) as f:
        return json.load(f)


def test_oracle_matches_stored_record():
    mk = _maker()
    stored = _stored()
    assert stored["case"] == mk.CASE and stored["rows"] == mk.ROWS
    now = mk.record(mk.compute())
    for name in ("LSE", "O", "dQ", "dK", "dV"):
        a, b = np.asarray(now[name]), np.asarray(stored[name])
        assert a.shape == b.shape, name
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12, err_msg=name)


def test_stored_record_closed_forms():
    stored = _stored()
    c = stored["case"]
    assert stored["rows"][0] == 0
    t = inputs.make_qkv(c["B"], c["H"], c["Hkv"], c["S"], c["D"], seed=c["seed"], with_do=True)
    q, k, v = (inputs.to_f64(t[n]) for n in ("q", "k", "v"))
    for h in range(c["H"]):
        g = h // (c["H"] // c["Hkv"])
        np.testing.assert_array_equal(np.asarray(stored["O"][h][0]), v[0, g, 0])
        assert abs(stored["LSE"][h][0] - c["scale"] * float(q[0, h, 0] @ k[0, g, 0])) < 1e-12
