"""Host logic of bench.py that needs no GPU: the parsers of the vendor SMI
tools' text (checked on output captured from an MI355X machine, idle) and the
refusal of more than one GPU."""
import os
import subprocess
import sys

import bench

HERE = os.path.dirname(os.path.abspath(__file__))


def _sample(name):
    with open(os.path.join(HERE, "tool_output", name)) as f:
        return f.read()


def test_parse_smi_metric_takes_socket_power_and_the_eight_xcd_clocks():
    watts, clks = bench.parse_smi_metric(_sample("amd_smi_metric_idle.txt"))
    assert watts == 268.0
    # GFX_0 .. GFX_7 only: the memory, video and SoC clocks of the same
    # listing (2000, 59, 48 and 40 MHz) are not shader clocks
    assert clks == [127, 125, 121, 120, 121, 121, 128, 127]


def test_parse_smi_metric_without_the_fields():
    assert bench.parse_smi_metric("") == (None, [])
    assert bench.parse_smi_metric("GPU: 0\n    POWER: N/A\n") == (None, [])


def test_parse_power_cap():
    assert bench.parse_power_cap(_sample("rocm_smi_maxpower.txt")) == 1400.0
    assert bench.parse_power_cap("no such field") is None


def test_more_than_one_gpu_is_refused():
    root = os.path.dirname(HERE)
    res = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=120)
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""
