"""CPU checks of the measurement contract.

* ``bench.py --gpus N`` with N > 1 refuses before touching a GPU (one GPU is
  all this library measures).
* The committed counter summaries describe the current kernels: every
  kernel's traffic entry in profiles/traffic.json carries the sha256 of its
  sources, and every profile names the current device-code hash, so a kernel
  changed without new profiles fails here (the bench would otherwise report
  its traffic as null).
"""
import json
import os
import re
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in (r.stdout + r.stderr)


def test_profiles_match_the_kernel_sources():
    t = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    for key, entry in t["kernels"].items():
        assert entry["source"] == bench.KERNEL_SOURCES[key]
        assert entry["source_sha256"] == bench._source_hash(entry["source"]), \
            f"{key}: kernel sources changed since the counters were taken"
    current = bench._kernel_source_hash()
    for name in os.listdir(os.path.join(ROOT, "profiles")):
        if name.endswith(".md"):
            text = open(os.path.join(ROOT, "profiles", name)).read()
            m = re.search(r"Kernel sources: sha256 ([0-9a-f]{64})", text)
            assert m and m.group(1) == current, f"{name} was made from other kernel sources"
