"""bench.py's host-side arithmetic (CPU): the rotation-calculus fit recovers the
model it assumes, the measured crossover is where the fused speedup crosses 1,
and the committed HBM traffic figure is used only while it matches the forward's
sources."""
import json
import math
from types import SimpleNamespace

import bench


def _sweep(a, b, c, sizes):
    """Synthetic sweep that follows the model exactly: no-RoPE time c S^2, fused
    time (a + c) S^2, separate rotation b S."""
    out = []
    for S in sizes:
        n, f, r = c * S * S, (a + c) * S * S, b * S
        out.append({"S": S, "fused_ms": f, "rope_ms": r, "norope_ms": n, "fused_speedup": (r + n) / f})
    return out


W = SimpleNamespace(B=1, H=32, Hkv=8, D=128)


def test_crossover_fit_recovers_the_model():
    a, b, c = 2e-9, 5e-6, 7e-9
    fit = bench.crossover_fit(_sweep(a, b, c, (1024, 2048, 4096, 8192, 16384)), W)
    assert math.isclose(fit["a_ms_per_S2"], a, rel_tol=1e-12)
    assert math.isclose(fit["b_ms_per_S"], b, rel_tol=1e-12)
    assert fit["S_star_model"] == round(b / a)
    assert fit["fit_points_S"] == [4096, 8192, 16384]


def test_measured_crossover_interpolates_in_log_s():
    # speedup (b/S + c)/(a + c) - 1 changes sign at S = b / a = 2500
    a, b, c = 2e-9, 5e-6, 7e-9
    sw = _sweep(a, b, c, (1024, 2048, 4096, 8192))
    fit = bench.crossover_fit(sw, W)
    lo, hi = sw[1], sw[2]
    assert lo["fused_speedup"] > 1 > hi["fused_speedup"]
    assert lo["S"] < fit["S_star_measured"] < hi["S"]
    f = (lo["fused_speedup"] - 1) / (lo["fused_speedup"] - hi["fused_speedup"])
    assert fit["S_star_measured"] == round(math.exp(math.log(2048) + f * math.log(2)))


def test_no_measured_crossover_when_fused_always_wins():
    sw = _sweep(1e-12, 5e-6, 7e-9, (1024, 2048, 4096, 8192))
    fit = bench.crossover_fit(sw, W)
    assert all(r["fused_speedup"] > 1 for r in sw) and fit["S_star_measured"] is None


def test_fit_needs_two_points_past_the_threshold():
    assert bench.crossover_fit(_sweep(2e-9, 5e-6, 7e-9, (1024, 2048, 4096)), W) is None


def test_traffic_used_only_for_current_sources(tmp_path, monkeypatch):
    rec = {"workload": "llama3_8b_b1h32kv8s8192d128", "source_sha256": bench.fwd_source_hash(),
           "traffic_bytes_per_launch": 123456789}
    path = tmp_path / "traffic.json"
    path.write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(path))
    assert bench.measured_traffic("llama3_8b_b1h32kv8s8192d128") == 123456789
    assert bench.measured_traffic("another_workload") is None
    path.write_text(json.dumps(dict(rec, source_sha256="0" * 64)))
    assert bench.measured_traffic("llama3_8b_b1h32kv8s8192d128") is None
    path.write_text("not json")
    assert bench.measured_traffic("llama3_8b_b1h32kv8s8192d128") is None

