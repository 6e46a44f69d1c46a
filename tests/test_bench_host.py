"""Host-side logic of bench.py (no GPU): the one-GPU contract, the traffic
records it reads from the committed rocprofv3 summaries, and the algorithmic
work it divides by."""
import importlib.util
import json
import os
import re
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
WORKLOADS = ("mixtral", "qwen3", "dsv3_prefill", "dsv3_decode", "dsv3_prefill_w8a8",
             "dsv3_decode_w8a8")


def _bench():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_every_profile_carries_a_traffic_record():
    for w in WORKLOADS:
        text = open(os.path.join(ROOT, "profiles", f"kernels_{w}.md")).read()
        m = re.search(r"```json\n(\{.*?\})\n```", text, re.S)
        assert m, w
        rec = json.loads(m.group(1))
        assert rec["workload"] == w
        assert rec["traffic_bytes"] == rec["read_bytes"] + rec["write_bytes"] > 0
        assert re.fullmatch(r"[0-9a-f]{64}", rec["kernel_source_sha256"])


def test_traffic_is_withheld_when_the_kernel_sources_changed(monkeypatch):
    b = _bench()
    text = open(os.path.join(ROOT, "profiles", "kernels_dsv3_prefill.md")).read()
    rec = json.loads(re.search(r"```json\n(\{.*?\})\n```", text, re.S).group(1))
    monkeypatch.setattr(b, "kernel_source_sha256", lambda: rec["kernel_source_sha256"])
    assert b.measured_traffic("dsv3_prefill") == rec["traffic_bytes"]
    monkeypatch.setattr(b, "kernel_source_sha256", lambda: "0" * 64)
    assert b.measured_traffic("dsv3_prefill") is None
    assert b.measured_traffic("no_such_workload") is None


def test_algorithmic_work():
    b = _bench()
    T, H, I, E, k = 8, 256, 128, 4, 2
    counts = np.array([6, 0, 5, 5])
    R = int(counts.sum())
    d = dict(T=T, H=H, I=I, E=E, k=k, wdtype="bf16")
    a = b.algorithmic(d, counts)
    assert a["flops"] == 6.0 * R * H * I == a["gu_flops"] + a["dn_flops"]
    # three active experts: their weights once, x once, h written then read, out written
    assert a["gu_bytes"] == 3 * 2 * I * H * 2 + T * H * 2 + R * I * 2 + R * 4
    assert a["dn_bytes"] == 3 * H * I * 2 + R * I * 2 + T * H * 2 + R * 4
    f8 = b.algorithmic(dict(d, wdtype="fp8"), counts)
    scales = 3 * ((2 * I // 128) * (H // 128) + (H // 128) * (I // 128)) * 4
    assert f8["gu_bytes"] + f8["dn_bytes"] == (a["gu_bytes"] + a["dn_bytes"]
                                                - 3 * 3 * I * H + scales)
