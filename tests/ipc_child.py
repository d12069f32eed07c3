"""Child processes of the zero-copy sharing test (tests/test_gpu_ipc.py).

``export SEED``: fill a paged KV pool of 64 regions x 512 blocks x 32 KiB
(1 GiB, one allocation) with seeded bf16 values, export it with
tc_ipc_export, print one JSON line (the handle's bytes, the pool's SHA-256,
its shape) and keep the pool alive until a line arrives on stdin.

``import HANDLE_HEX SHA``: open the handle, gather 256 block ids of every
region straight out of the imported pool with tc_gather_blocks, and check
(1) that the imported bytes are the exporter's (SHA-256 of a copy) and
(2) that the gathered buffer equals the oracle's gather of those bytes.
Then time the same gather from the imported pool and from a local copy of
it, and print one JSON line with both rates.
"""
import ctypes
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

R, NB, B = 64, 512, 32768
N_IDS = 256


def _log(msg):
    print(msg, file=sys.stderr, flush=True)


def export(seed: int) -> int:
    import torch
    import synth
    import paper_2608_06007_amd as tc
    torch.cuda.set_device(0)
    pool = synth.bf16_normal(R * NB * B // 2, 1.0, seed, device="cuda").view(torch.uint8)
    torch.cuda.synchronize()
    handle = tc.tc_ipc_export(pool)
    sha = hashlib.sha256(pool.cpu().numpy().tobytes()).hexdigest()
    print(json.dumps({"handle": handle.hex(), "sha256": sha, "bytes": pool.numel()}), flush=True)
    _log("exporter: waiting for the importer")
    sys.stdin.readline()
    torch.cuda.synchronize()
    _log("exporter: done")
    return 0


def _hip_runtime():
    for name in ("libamdhip64.so", "/opt/rocm/lib/libamdhip64.so"):
        try:
            lib = ctypes.CDLL(name)
            lib.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
            lib.hipMemcpy.restype = ctypes.c_int
            return lib
        except OSError:
            continue
    raise RuntimeError("HIP runtime library not found")


def _gbps(torch, fn, nbytes, reps=20):
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ms = []
    for _ in range(reps):
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1))
    ms.sort()
    med = ms[len(ms) // 2]
    return round(nbytes / (med * 1e-3) / 1e9, 1), round(med, 4)


def import_(handle_hex: str, sha: str) -> int:
    import numpy as np
    import torch
    import oracle
    import synth
    import paper_2608_06007_amd as tc
    torch.cuda.set_device(0)
    handle = bytes.fromhex(handle_hex)
    base = tc.tc_ipc_open(handle)
    _log(f"importer: opened the pool at {base:#x}")
    region_bytes = NB * B
    regions = [base + r * region_bytes for r in range(R)]
    ids_np = synth.ids_without_replacement(NB, N_IDS, seed=1701)
    ids = torch.from_numpy(ids_np).cuda()
    out = torch.empty(N_IDS * R * B, dtype=torch.uint8, device="cuda")
    tc.tc_gather_blocks(regions, NB, B, B, ids, out)
    torch.cuda.synchronize()
    # the imported bytes, copied to the host by the runtime's own hipMemcpy
    host = np.empty(R * region_bytes, dtype=np.uint8)
    hip = _hip_runtime()
    rc = hip.hipMemcpy(ctypes.c_void_p(host.ctypes.data), ctypes.c_void_p(base),
                       ctypes.c_size_t(host.nbytes), 2)  # hipMemcpyDeviceToHost
    if rc != 0:
        _log(f"importer: hipMemcpy of the imported pool failed ({rc})")
        return 2
    if hashlib.sha256(host.tobytes()).hexdigest() != sha:
        _log("importer: the imported bytes are not the exporter's")
        return 3
    local = torch.from_numpy(host).cuda()
    local_regions = [local[r * region_bytes:(r + 1) * region_bytes] for r in range(R)]
    want = oracle.gather_blocks([host[r * region_bytes:(r + 1) * region_bytes] for r in range(R)],
                                B, B, ids_np)
    if not np.array_equal(out.cpu().numpy(), want.reshape(-1)):
        _log("importer: gather from the imported pool differs from the oracle")
        return 4
    nbytes = 2 * N_IDS * R * B
    imp, imp_ms = _gbps(torch, lambda: tc.tc_gather_blocks(regions, NB, B, B, ids, out), nbytes)
    loc, loc_ms = _gbps(torch, lambda: tc.tc_gather_blocks(local_regions, NB, B, B, ids, out), nbytes)
    tc.tc_ipc_close(handle, base)
    print(json.dumps({"ok": True, "gather_bytes": nbytes, "imported_GBps": imp, "imported_ms": imp_ms,
                      "local_GBps": loc, "local_ms": loc_ms}), flush=True)
    return 0


if __name__ == "__main__":
    if sys.argv[1] == "export":
        sys.exit(export(int(sys.argv[2])))
    sys.exit(import_(sys.argv[2], sys.argv[3]))
