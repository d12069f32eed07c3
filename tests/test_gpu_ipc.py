"""GPU: zero-copy sharing of a device KV pool between two processes on one
GPU through HIP IPC (the Unified Tensor Pool's same-host sharing, Sec. 4.2
and Sec. 5; the warm start's zero-copy consumption, Sec. 6.1).

An exporter process fills a 1 GiB paged KV pool and publishes its handle; an
importer process opens it, checks that the mapped bytes are the exporter's
(the runtime's own hipMemcpy, SHA-256), gathers 256 block ids straight out of
the imported pool and compares the result with the oracle's gather of those
bytes.  Both are fresh processes (tests/ipc_child.py); this process only
starts them, passes the handle and waits.
"""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CHILD = os.path.join(ROOT, "tests", "ipc_child.py")


def _env():
    env = dict(os.environ)
    # one allocation per tensor, so the exported pool is an allocation of its own
    env["PYTORCH_NO_CUDA_MEMORY_CACHING"] = "1"
    env["PYTORCH_NO_HIP_MEMORY_CACHING"] = "1"
    env.setdefault("HSA_ENABLE_IPC_MODE_LEGACY", "0")
    return env


def test_ipc_export_and_gather_from_another_process():
    print("case: IPC export (1 GiB KV pool) -> import + gather of 256 ids", flush=True)
    exporter = subprocess.Popen([sys.executable, "-u", CHILD, "export", "1702"], stdin=subprocess.PIPE,
                                stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True, env=_env())
    try:
        line = exporter.stdout.readline()
        assert line, "exporter ended early: " + exporter.stderr.read()
        info = json.loads(line)
        assert info["bytes"] == 1 << 30
        imp = subprocess.run([sys.executable, "-u", CHILD, "import", info["handle"], info["sha256"]],
                             capture_output=True, text=True, env=_env(), timeout=90)
        print(imp.stderr, flush=True)
        assert imp.returncode == 0, f"importer failed ({imp.returncode}): {imp.stderr[-2000:]}"
        res = json.loads(imp.stdout.strip().splitlines()[-1])
        assert res["ok"]
        print(f"gather of {res['gather_bytes']} B: imported pool {res['imported_GBps']} GB/s, "
              f"local copy {res['local_GBps']} GB/s", flush=True)
        exporter.stdin.write("done\n")
        exporter.stdin.flush()
        assert exporter.wait(timeout=60) == 0, exporter.stderr.read()
    finally:
        if exporter.poll() is None:
            exporter.kill()
            exporter.wait()
