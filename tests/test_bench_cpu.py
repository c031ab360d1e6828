"""bench.py's host-side pieces, checked on the CPU.

- The kernel-code hash ignores comments and whitespace, and changes with
  the code.
- The committed HBM-traffic record of the benchmark's history launch was
  taken on the current kernel code, so the benchmark line reports it; its
  arithmetic (copy-calibrated counters over the algorithmic bytes) holds.
- The kernel-trace, traffic and utilisation summaries under profiles/
  name the same kernel code.
- A run asked for more than one GPU exits with a message before touching
  any GPU.
"""
from __future__ import annotations

import importlib.util
import json
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_code_hash_ignores_comments_and_whitespace():
    b = _bench()
    src = "int f(int x) {\n  return x + 1;  // one\n}\n"
    assert b.code_hash(src) == b.code_hash("/* header */\nint f(int x)\n{ return x+1; }\n// trailing\n")
    assert b.code_hash(src) != b.code_hash(src.replace("x + 1", "x + 2"))


def test_traffic_record_matches_the_current_kernel():
    b = _bench()
    with open(b.TRAFFIC_FILE) as f:
        tr = json.load(f)
    assert tr["kernel_code_sha256_16"] == b.kernel_source_hash(), \
        "profiles/chunk_attn_config3_traffic.json was taken on other kernel code: collect the counters again"
    assert tr["config"] == 3 and tr["kv_layout"] == "head-kv"
    cal = tr["copy_calibration"]
    # the calibration factors are the copy's true bytes over what the counters read
    assert abs(cal["bytes_copied"] / 1024 / cal["fetch_size_kib"] - cal["fetch_factor"]) < 0.01
    assert abs(cal["bytes_copied"] / 1024 / cal["write_size_kib"] - cal["write_factor"]) < 0.01
    hbm = (tr["fetch_size_kib_per_launch"] * cal["fetch_factor"] + tr["write_size_kib_per_launch"] * cal["write_factor"]) * 1024
    assert abs(hbm - tr["hbm_bytes_per_launch"]) <= 1024
    assert tr["algorithmic_bytes_per_launch"] == 16 * 32768 * 8 * 128 * 2 * 2
    assert abs(tr["hbm_bytes_per_launch"] / tr["algorithmic_bytes_per_launch"] - tr["traffic_over_algorithmic"]) < 1e-4
    # every K/V byte read once, plus the query rows and the state slots
    assert 1.0 <= tr["traffic_over_algorithmic"] < 1.02


def test_profile_summaries_name_the_current_kernel():
    b = _bench()
    h = b.kernel_source_hash()
    for name in ("chunk_attn_config3_kernel_trace.md", "chunk_attn_config3_traffic.md", "chunk_attn_config5_traffic.md",
                 "chunk_attn_utilisation.md", "chunk_attn_wide_64rows_config3_shape.md"):
        with open(os.path.join(ROOT, "profiles", name)) as f:
            text = f.read()
        found = set(re.findall(r"`([0-9a-f]{16})`", text))
        assert found == {h}, f"profiles/{name} names kernel code {sorted(found)}, the source is {h}"


def test_more_than_one_gpu_is_refused():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                         text=True, timeout=120, cwd=ROOT)
    assert res.returncode == 2
    assert "one GPU only" in res.stderr
    assert res.stdout == ""
