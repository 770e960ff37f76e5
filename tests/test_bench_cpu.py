"""Host-side checks of bench.py's contract (no GPU needed)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_is_refused(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_clock_sampler_without_sysfs(monkeypatch):
    import glob
    import bench
    monkeypatch.setattr(glob, "glob", lambda pattern: [])
    with bench.ClockSampler(period_s=0.001) as c:
        pass
    assert c.path is None and c.power_path is None
    assert c.summary() is None and c.power_summary() is None


def test_clock_sampler_reads_fake_sysfs(tmp_path, monkeypatch):
    import glob
    import time
    import bench
    dev = tmp_path / "card0" / "device"
    hw = dev / "hwmon" / "hwmon0"
    hw.mkdir(parents=True)
    (dev / "pp_dpm_sclk").write_text("0: 500Mhz\n1: 1750Mhz *\n2: 2400Mhz\n")
    (hw / "power1_input").write_text("1377000000\n")
    (hw / "power1_cap").write_text("1400000000\n")
    real_glob = glob.glob

    def fake(pattern):
        if pattern.startswith("/sys/class/drm/"):
            return sorted(real_glob(pattern.replace("/sys/class/drm", str(tmp_path))))
        return real_glob(pattern)

    monkeypatch.setattr(glob, "glob", fake)
    with bench.ClockSampler(period_s=0.001) as c:
        time.sleep(0.05)
    s, p = c.summary(), c.power_summary()
    assert s["mean"] == 1750.0 and s["samples"] >= 1
    assert p["mean"] == pytest.approx(1377.0) and p["cap"] == pytest.approx(1400.0)
