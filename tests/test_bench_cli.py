"""bench.py host logic (no GPU): the one-GPU guard, the clock and temperature reading, the oracle sample size."""

import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


def test_sysfs_reading(tmp_path, monkeypatch):
    """The starred level of pp_dpm_sclk is the clock; the hottest hwmon sensor the temperature."""
    import glob as g

    dev = tmp_path / "card0" / "device"
    (dev / "hwmon" / "hwmon3").mkdir(parents=True)
    (dev / "pp_dpm_sclk").write_text("0: 500Mhz\n1: 1991Mhz *\n2: 2400Mhz\n")
    (dev / "hwmon" / "hwmon3" / "temp1_input").write_text("41000\n")
    (dev / "hwmon" / "hwmon3" / "temp2_input").write_text("52500\n")
    real = g.glob

    def fake(pat, *a, **k):
        return real(pat.replace("/sys/class/drm", str(tmp_path)), *a, **k)

    monkeypatch.setattr(g, "glob", fake)
    assert bench.sysfs_reading() == (1991.0, 52.5)


def test_cpu_sample_b():
    # the whole batch when the oracle's estimate is under 40 s, else a multiple of 4096 near 20 s
    assert bench.cpu_sample_b(32768, 512) == 32768
    assert bench.cpu_sample_b(131072, 768) == 20480
    assert bench.cpu_sample_b(1 << 22, 768) % 4096 == 0
