"""GPU: the two measurement programs that build() puts next to the library
(streaming ceiling of the context ring; L2 hand-off between launches) run on
the device and report figures in range.  They are measurement tools, not part
of the library's API."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.gpu


def _run(name: str, timeout: int) -> str:
    exe = os.path.join(ROOT, "paper_2609_05707_amd", name)
    if not os.path.exists(exe):
        pytest.skip(f"{name} is not built (build() builds it next to libippd.so)")
    print(f"case: {name}", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=timeout)
    assert r.returncode == 0, r.stderr[-2000:]
    return r.stdout


def test_stream_ceiling_reports_ring_and_register_loads():
    out = _run("stream_ceiling", 120)
    rates = {m.group(1): float(m.group(2))
             for m in re.finditer(r"^\s*(ring|loads)\s+268435456\s+[\d.]+\s+([\d.]+)\s", out, re.M)}
    assert set(rates) == {"ring", "loads"}, out
    # GB/s: well above a stalled stream, below the 8 TB/s HBM peak
    assert all(1000.0 < v < 8000.0 for v in rates.values()), rates


def test_l2_handoff_reports_each_reader_placement():
    out = _run("l2_handoff", 60)
    rows = re.findall(r"reader on XCD (\d), writer on XCD 0: ([\d.]+) us per 2 MiB read", out)
    assert [int(x) for x, _ in rows] == [0, 1, 0, 1], out
    assert all(0.0 < float(us) < 1000.0 for _, us in rows), rows
