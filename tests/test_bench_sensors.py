"""bench.py's power and clock sampler reads sysfs files only; its parsing is
checked here on a fake sysfs tree (CPU)."""
import os
import sys
import time

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _tree(tmp_path, sclk, power_uw, cap_uw):
    dev = tmp_path / "card0" / "device"
    (dev / "hwmon" / "hwmon3").mkdir(parents=True)
    (dev / "pp_dpm_sclk").write_text(sclk)
    (dev / "hwmon" / "hwmon3" / "power1_input").write_text(f"{power_uw}\n")
    (dev / "hwmon" / "hwmon3" / "power1_cap").write_text(f"{cap_uw}\n")
    return dev


def test_sampler_reads_power_cap_and_marked_clock(tmp_path):
    _tree(tmp_path, "0: 500Mhz\n1: 2400Mhz *\n", 1234500000, 1400000000)
    with bench.GpuSensors(period=0.005, root=str(tmp_path)) as s:
        time.sleep(0.05)
    out = s.summary()
    assert out["gpu_sensor_samples"] >= 2
    assert out["gpu_power_w_mean"] == 1234.5 and out["gpu_power_w_max"] == 1234.5
    assert out["gpu_power_cap_w"] == 1400.0
    assert out["gpu_sclk_mhz_median"] == 2400


def test_sampler_reads_the_deep_sleep_line(tmp_path):
    _tree(tmp_path, "S: 95Mhz *\n0: 500Mhz\n1: 2400Mhz\n", 235000000, 1400000000)
    with bench.GpuSensors(period=0.005, root=str(tmp_path)) as s:
        time.sleep(0.03)
    assert s.summary()["gpu_sclk_mhz_median"] == 95


def test_sampler_without_files_reports_none(tmp_path):
    with bench.GpuSensors(period=0.005, root=str(tmp_path)) as s:
        time.sleep(0.01)
    out = s.summary()
    assert out["gpu_sensor_samples"] == 0
    assert all(out[k] is None for k in ("gpu_power_w_mean", "gpu_power_w_max", "gpu_power_cap_w", "gpu_sclk_mhz_median"))
