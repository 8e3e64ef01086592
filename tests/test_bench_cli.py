"""bench.py host logic (no GPU): the one-GPU guard and the rocm-smi reading."""

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


def test_smi_reading():
    text = ('{"card0": {"Temperature (Sensor edge) (C)": "40.0", "Temperature (Sensor junction) (C)": "52.0", '
            '"mclk clock speed:": "(1900Mhz)", "sclk clock speed:": "(2400Mhz)"}}')
    assert bench.smi_reading(text) == (2400.0, 52.0)
    # edge temperature when no junction sensor is listed
    assert bench.smi_reading('{"card0": {"Temperature (Sensor edge) (C)": "41.5"}}') == (None, 41.5)
    assert bench.smi_reading("not json") == (None, None)
    assert bench.smi_reading("{}") == (None, None)
