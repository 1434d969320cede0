"""Host logic of bench.py (no GPU): the roofline fractions it reports and
the gate on its stored HBM-traffic figures, which hold only for the kernel
sources they were measured on."""

import copy

import pytest

import bench


def test_rate_fractions():
    # 304 MB and 34.4 GFLOP in 0.0625 ms: HBM-bound, binding fraction = HBM fraction
    r = bench.rate(304_070_656, 34_359_738_368, 0.0625)
    assert r["gbs"] == pytest.approx(304_070_656 / 0.0625e-3 / 1e9, rel=1e-3)
    assert r["frac_hbm"] == pytest.approx(r["gbs"] / bench.HBM_PEAK_GBS, abs=1e-4)
    assert r["frac_binding"] == r["frac_hbm"]
    # 2.474 TFLOP over 436 MB in 2 ms: MFMA-bound, binding fraction = MFMA fraction
    r = bench.rate(436_207_616, 2_474_035_380_224, 2.0)
    assert r["tflops"] == pytest.approx(1237.02, abs=0.01)
    assert r["frac_binding"] == r["frac_mfma"]
    # bytes only: no MFMA or binding entries
    assert set(bench.rate(1 << 30, ms=1.0)) == {"gbs", "frac_hbm"}


@pytest.mark.parametrize("key", sorted(bench.MEASURED_TRAFFIC))
def test_stored_traffic_matches_current_sources(key):
    """Each stored FETCH+WRITE figure was measured on the kernel sources as they
    are now (re-measure with the rocprofv3 passes of the traffic profile
    after changing a kernel, and update the figure and its SHA-256)."""
    b = bench.measured_traffic(key)
    assert b is not None, f"{key}: kernel sources changed since their traffic was measured"
    assert b > 0


def test_traffic_gate_rejects_changed_sources(monkeypatch):
    table = copy.deepcopy(bench.MEASURED_TRAFFIC)
    table["prefill_full"]["sha256"] = "0" * 64
    monkeypatch.setattr(bench, "MEASURED_TRAFFIC", table)
    assert bench.measured_traffic("prefill_full") is None
