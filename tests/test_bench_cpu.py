"""Host-side pieces of bench.py: reading the committed rocprofv3 summaries.

The roofline's `traffic` and `hardware_fraction` come from the machine-readable
block of a profile only while its recorded kernel source hash matches the
current source; a stale or missing summary gives None, never old figures."""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _write_profile(tmp_path, fields):
    d = tmp_path / "profiles"
    d.mkdir(exist_ok=True)
    body = "# summary\n\n```json\n" + json.dumps(fields, indent=1) + "\n```\n"
    (d / "k_simulate_amin_wl.md").write_text(body)


def test_current_profile_fields(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "x")
    _write_profile(tmp_path, {"kernel_source_hash": "x", "hbm_bytes_per_launch": 123, "valu_busy_pct": 25.0,
                              "valu_utilization_pct": 80.0, "lds_bank_conflict_pct": 0.05})
    assert bench.load_traffic("wl", "amin") == 123
    hw = bench.load_hardware_fraction("wl", "amin")
    assert abs(hw["valu_lane_cycles"] - 0.2) < 1e-12
    assert hw["lds_bank_conflict_pct"] == 0.05
    assert "lds_frac_max" not in hw           # no LDS instruction count in this summary


def test_lds_bound_from_instruction_count(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "x")
    _write_profile(tmp_path, {"kernel_source_hash": "x", "hbm_bytes_per_launch": 1, "valu_busy_pct": 10.0,
                              "valu_utilization_pct": 50.0, "lds_insts_per_launch": 1e6})
    hw = bench.load_hardware_fraction("wl", "amin", kernel_ms=2.0)
    # 1e6 wave64 instructions x 8 B x 64 lanes over 2 ms, against 256 CUs x 128 B x 2.4 GHz
    assert hw["lds_bytes_per_launch_max"] == 1e6 * 512
    assert abs(hw["lds_frac_max"] - (512e6 / 2e-3) / (256 * 128 * 2.4e9)) < 1e-15


def test_stale_or_missing_profile_gives_none(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "current")
    assert bench.load_traffic("wl", "amin") is None          # no file
    _write_profile(tmp_path, {"kernel_source_hash": "older", "hbm_bytes_per_launch": 5,
                              "valu_busy_pct": 1.0, "valu_utilization_pct": 1.0})
    assert bench.load_traffic("wl", "amin") is None
    assert bench.load_hardware_fraction("wl", "amin") is None


def test_committed_profiles_parse():
    # the summaries bench reads (k_simulate_<policy>_<workload>.md) carry a
    # parseable block with the fields it uses
    d = os.path.join(ROOT, "profiles")
    policies = ("amin", "amax", "hsf", "aell", "adaptive", "arandom")
    read = [n for n in os.listdir(d) if any(n.startswith(f"k_simulate_{a}_") for a in policies)]
    assert "k_simulate_amin_batch4096_n1000_m16384.md" in read
    for name in read:
        text = open(os.path.join(d, name)).read()
        block = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
        assert isinstance(block["kernel_source_hash"], str)
        # every summary has the lane-cycle figures; the benchmark's also the traffic
        assert block["valu_busy_pct"] >= 0 and block["valu_utilization_pct"] >= 0
        if name == "k_simulate_amin_batch4096_n1000_m16384.md":
            assert block["hbm_bytes_per_launch"] > 0
