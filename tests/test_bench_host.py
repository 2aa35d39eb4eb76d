"""Host-side logic of bench.py (no GPU): the one-GPU guard, the amdsmi
reader's device matching and averaging (with a stand-in module), and the
trace summary's pass selection and arithmetic on a synthetic kernel trace."""
import json
import os
import subprocess
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


def _fake_amdsmi(metrics, bdfs):
    m = types.ModuleType("amdsmi")
    m.amdsmi_init = lambda: None
    m.amdsmi_get_processor_handles = lambda: list(range(len(bdfs)))
    m.amdsmi_get_gpu_device_bdf = lambda h: bdfs[h]
    m.amdsmi_get_gpu_metrics_info = lambda h: metrics[h]
    return m


def test_sensors_match_the_device_by_pci_address(monkeypatch):
    props = types.SimpleNamespace(pci_domain_id=0, pci_bus_id=0x75, pci_device_id=0)
    monkeypatch.setattr(bench.torch.cuda, "get_device_properties", lambda i: props)
    metrics = [{"current_gfxclks": [100] * 8, "current_socket_power": 200, "temperature_hotspot": 40},
               {"current_gfxclks": [1900, 1910, 1920, 1930, "N/A", 1950, 1960, 1970],
                "current_socket_power": 1300, "temperature_hotspot": "N/A"}]
    monkeypatch.setitem(sys.modules, "amdsmi",
                        _fake_amdsmi(metrics, ["0000:05:00.0", "0000:75:00.0"]))
    s = bench.GpuSensors(0)
    assert s.handle == 1
    r = s.sample()
    assert r == {"gfx_mhz": round(sum([1900, 1910, 1920, 1930, 1950, 1960, 1970]) / 7, 1),
                 "power_w": 1300, "hotspot_c": None}


def test_sensors_report_nothing_without_a_match_or_amdsmi(monkeypatch):
    props = types.SimpleNamespace(pci_domain_id=0, pci_bus_id=0x11, pci_device_id=0)
    monkeypatch.setattr(bench.torch.cuda, "get_device_properties", lambda i: props)
    monkeypatch.setitem(sys.modules, "amdsmi", _fake_amdsmi([{}], ["0000:05:00.0"]))
    assert bench.GpuSensors(0).sample() is None
    monkeypatch.setitem(sys.modules, "amdsmi", None)     # import fails
    assert bench.GpuSensors(0).sample() is None


def test_trace_summary_takes_the_timed_and_events_passes(tmp_path):
    """Chunks 2 + 1, warm-up 2 and 3 timed steps: dispatches 0-3 warm-up,
    4-9 timed, 10-15 the events pass.  Each launch of h heads lasts h ms in
    the timed steps and h + 0.01 ms in the events pass; the warm-up launches
    are slower and must be left out."""
    S, d, chunks, W, K = 56160, 128, [2, 1], 2, 3
    rows, t = [], 0
    for step in range(W + 2 * K):
        for h in chunks:
            dur = {True: 5.0 * h}.get(step < W, h + (0.01 if step >= W + K else 0.0))
            rows.append((t, t + int(round(dur * 1e6))))
            t += int(round(dur * 1e6)) + 1000
    csv_path = tmp_path / "trace.csv"
    with open(csv_path, "w") as f:
        f.write("Kernel_Name,Start_Timestamp,End_Timestamp\n")
        f.write("pack_kernel,0,1\n")
        for b, e in rows:
            f.write(f"attention_dma_kernel<true>,{b},{e}\n")
    flops = 4.0 * S * S * d * sum(chunks) * K
    ach = flops / (sum(chunks) * K * 1e-3) / 1e12
    line = {"metric": "m", "value": 1.0, "ms_per_step": 3.05, "warmup": W, "steps": K,
            "config": {"chunks": chunks, "S": S, "d": d, "workload": "w"},
            "roofline": {"achieved": round(ach, 2), "frac": round(ach / bench.MFMA_BF16_PEAK_TFLOPS, 4),
                         "events_pass": {"frac": 0.5}}}
    line_path = tmp_path / "line.json"
    line_path.write_text("log line\n" + json.dumps(line) + "\n")
    out = bench.trace_summary(str(csv_path), str(line_path))
    assert "Attention dispatches in the trace: 16." in out
    assert f"| timed steps | 4..9 | {1.5:.4f} | {3.0:.4f} | {ach:.1f} |" in out
    ev = flops / ((sum(chunks) + 0.02) * K * 1e-3) / 1e12
    assert f"| {(3.02 / 2):.4f} | {3.02:.4f} | {ev:.1f} |" in out
    assert "<= the line's ms_per_step 3.05: True." in out
    import re
    apart = re.search(r"timed steps 0\.6417 against the line's 0\.6417: ([0-9.]+) % apart", out)
    assert apart and float(apart.group(1)) < 0.02     # the line's frac is rounded to 4 places
    with pytest.raises(SystemExit):
        (tmp_path / "empty.json").write_text("no line\n")
        bench.trace_summary(str(csv_path), str(tmp_path / "empty.json"))
