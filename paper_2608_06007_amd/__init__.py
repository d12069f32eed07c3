"""MI355X (gfx950) data path beneath TensorCast's tensor lifecycle primitives.

A thin ctypes binding over ``libtchip.so`` (built from ``csrc/`` by
``build.py``).  The functions keep the C ABI's names and only marshal
arguments: torch tensors supply device memory and streams, and every byte
the path moves is moved by the library's HIP kernels.  There is no CPU
fallback: if the library is missing, every call raises.

Entry points (see include/tensorcast_hip.h for the contracts):

* ``tc_gather_blocks`` / ``tc_scatter_blocks`` -- publish / hydrate of a
  request's paged KV blocks (paper Sec. 3.2 "Operation", Table 2).
* ``tc_copy_fragments`` (+ ``tc_plan_fragments`` / ``tc_copy_planned``) --
  batched byte fragments, as in prefetch_many and the materialization
  transfer stage (Table 2, Sec. 5).
* ``tc_copy_planned_digest`` / ``tc_digest_planned`` -- the same copies with
  a per-fragment integrity digest (the verify stage of Sec. 5).
* ``tc_stager_create`` ... ``tc_hydrate_from_host`` / ``tc_publish_to_host`` --
  pinned-ring staging between host memory and the device (Sec. 5).
* ``tc_tp_fragments`` / ``tc_tp_cast_item`` -- host builders that describe a
  tensor-parallel rank's view(slice) of each weight (Table 2, Sec. 6.1-6.2).
* ``tc_cast_fp8_blockscaled`` (+ ``tc_cast_fp8_prepare`` /
  ``tc_cast_fp8_planned``) / ``tc_cast_fp8_scaled`` -- a transform_into rule:
  bf16 -> fp8 E4M3 with an fp32 scale per 128x128 tile; and its inverse,
  ``tc_dequant_fp8_blockscaled`` (+ prepare / planned).
* ``tc_ipc_export`` / ``tc_ipc_open`` / ``tc_ipc_close`` -- zero-copy sharing
  of device ranges between processes on one host (Sec. 4.2, Sec. 5).
"""
from __future__ import annotations

import ctypes
import os
import sys as _sys

import numpy as np

__all__ = [
    "TcError", "lib_path", "load",
    "tc_gather_blocks", "tc_scatter_blocks",
    "tc_copy_fragments_workspace", "tc_copy_fragments_workspace_min", "tc_copy_fragments", "tc_plan_fragments",
    "tc_plan_fragments_async", "tc_plan_status", "tc_copy_planned", "TASKS_FROM_PLAN",
    "tc_copy_planned_digest", "tc_digest_planned", "DIGEST_SRC", "DIGEST_DST",
    "tc_tp_fragment_count", "tc_tp_fragments", "tc_tp_cast_item",
    "tc_reshard_fragment_count", "tc_reshard_fragments",
    "tc_reshard_cast_item_count", "tc_reshard_cast_items",
    "tc_cast_fp8_workspace", "tc_cast_fp8_workspace_tiles", "tc_cast_fp8_blockscaled", "tc_cast_fp8_scaled",
    "tc_cast_fp8_prepare", "tc_cast_fp8_planned", "TilePlan",
    "tc_dequant_fp8_workspace", "tc_dequant_fp8_workspace_tiles", "tc_dequant_fp8_blockscaled",
    "DEQUANT_ITEM_DTYPE",
    "tc_dequant_fp8_prepare", "tc_dequant_fp8_planned",
    "tc_ipc_export", "tc_ipc_open", "tc_ipc_close", "IPC_HANDLE_BYTES",
    "tc_stager_create", "tc_stager_destroy", "tc_stage_h2d", "tc_stage_d2h",
    "tc_hydrate_from_host", "tc_publish_to_host", "Stager", "HOST_PINNED",
    "tc_status_string", "tc_last_hip_error", "tc_set_validate", "tc_get_validate",
    "FRAGMENT_DTYPE", "TP_VIEW_DTYPE", "CAST_ITEM_DTYPE",
    "SPLIT_NONE", "SPLIT_ROWS", "SPLIT_COLS", "MAX_REGIONS",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
# TC_LIB_PATH loads another build of the same library (the CPU test tier runs
# the host code under sanitizers that way).
lib_path = os.environ.get("TC_LIB_PATH") or os.path.join(_HERE, "libtchip.so")

MAX_REGIONS = 256
SPLIT_NONE, SPLIT_ROWS, SPLIT_COLS = 0, 1, 2
DIGEST_SRC, DIGEST_DST = 0, 1
HOST_PINNED = 1
TASKS_FROM_PLAN = (1 << 64) - 1   # tc_copy_planned: the count is read from the plan on the device
TC_OK = 0
_STATUS = {0: "TC_OK", 1: "TC_ERR_INVALID_ARGUMENT", 2: "TC_ERR_OUT_OF_RANGE", 3: "TC_ERR_ALIAS",
           4: "TC_ERR_HIP", 5: "TC_ERR_WORKSPACE", 6: "TC_ERR_HOST_RESOURCES"}

# Host layouts of the C structs.
FRAGMENT_DTYPE = np.dtype([("src_off", "<u8"), ("dst_off", "<u8"), ("len", "<u8")])
TP_VIEW_DTYPE = np.dtype([("src_off", "<u8"), ("rows", "<i8"), ("cols", "<i8"), ("src_ld", "<i8"),
                          ("dst_off", "<u8"), ("dst_ld", "<i8"), ("elem_bytes", "<i4"),
                          ("split", "<i4")])
DEQUANT_ITEM_DTYPE = np.dtype([("src_off", "<u8"), ("rows", "<i8"), ("cols", "<i8"), ("src_ld", "<i8"),
                               ("dst_off", "<u8"), ("dst_ld", "<i8"), ("scale_off", "<u8"),
                               ("scale_ld", "<i8")])
CAST_ITEM_DTYPE = np.dtype([("src_off", "<u8"), ("rows", "<i8"), ("cols", "<i8"), ("src_ld", "<i8"),
                            ("dst_off", "<u8"), ("dst_ld", "<i8"), ("scale_off", "<u8"),
                            ("scale_ld", "<i8")])


class TcError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        name = _STATUS.get(status, str(status))
        extra = ""
        if status == 4:
            extra = f" (hipError {load().tc_last_hip_error()})"
        super().__init__(f"{what}: {name}{extra}")


class _ReshardView(ctypes.Structure):
    _fields_ = [("src_off", ctypes.POINTER(ctypes.c_uint64)), ("rows", ctypes.c_int64),
                ("cols", ctypes.c_int64), ("elem_bytes", ctypes.c_int32), ("split", ctypes.c_int32),
                ("src_tp", ctypes.c_int32), ("reserved", ctypes.c_int32), ("dst_off", ctypes.c_uint64)]


class TilePlan(ctypes.Structure):
    """tc_tile_plan: a cast (or inverse-cast) tile table prepared in a workspace."""
    _fields_ = [("n_items", ctypes.c_int64), ("full_tiles", ctypes.c_uint64),
                ("edge_tiles", ctypes.c_uint64), ("in_align", ctypes.c_uint32),
                ("out_align", ctypes.c_uint32), ("tiled", ctypes.c_uint32),
                ("reserved", ctypes.c_uint32)]


class _IpcHandle(ctypes.Structure):
    _fields_ = [("handle", ctypes.c_uint8 * 64), ("offset", ctypes.c_uint64), ("bytes", ctypes.c_uint64),
                ("alloc_bytes", ctypes.c_uint64)]


IPC_HANDLE_BYTES = ctypes.sizeof(_IpcHandle)


class _BlockPool(ctypes.Structure):
    _fields_ = [("region_base", ctypes.POINTER(ctypes.c_uint64)), ("num_regions", ctypes.c_int32),
                ("num_blocks", ctypes.c_int64), ("block_bytes", ctypes.c_int64),
                ("block_stride", ctypes.c_int64)]


_lib = None


def load():
    """Load libtchip.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(lib_path):
        raise RuntimeError(f"{lib_path} is missing: build it with paper_2608_06007_amd/build.py")
    L = ctypes.CDLL(lib_path)
    c = ctypes
    P = c.c_void_p
    L.tc_gather_blocks.argtypes = [c.POINTER(_BlockPool), P, c.c_int64, P, P]
    L.tc_scatter_blocks.argtypes = [c.POINTER(_BlockPool), P, c.c_int64, P, P]
    L.tc_copy_fragments_workspace.argtypes = [c.c_int64]
    L.tc_copy_fragments_workspace.restype = c.c_size_t
    L.tc_copy_fragments_workspace_min.argtypes = [c.c_int64]
    L.tc_copy_fragments_workspace_min.restype = c.c_size_t
    L.tc_copy_fragments.argtypes = [P, P, P, c.c_int64, P, c.c_size_t, P]
    L.tc_plan_fragments.argtypes = [P, c.c_int64, P, c.c_size_t, c.POINTER(c.c_uint64), P]
    L.tc_copy_planned.argtypes = [P, P, P, c.c_size_t, c.c_uint64, P]
    L.tc_plan_fragments_async.argtypes = [P, c.c_int64, P, c.c_size_t, P]
    L.tc_plan_status.argtypes = [P, c.c_size_t, c.POINTER(c.c_uint64), P]
    L.tc_copy_planned_digest.argtypes = [P, P, P, c.c_size_t, c.c_uint64, c.c_int64, P, P]
    L.tc_digest_planned.argtypes = [P, c.c_int32, P, c.c_size_t, c.c_uint64, c.c_int64, P, P]
    L.tc_tp_fragment_count.argtypes = [P, c.c_int64, c.c_int32, c.c_int32]
    L.tc_tp_fragment_count.restype = c.c_int64
    L.tc_tp_fragments.argtypes = [P, c.c_int64, c.c_int32, c.c_int32, P, c.c_int64,
                                  c.POINTER(c.c_int64)]
    L.tc_tp_cast_item.argtypes = [P, c.c_int32, c.c_int32, c.c_uint64, P]
    L.tc_reshard_fragment_count.argtypes = [P, c.c_int64, c.c_int32, c.c_int32]
    L.tc_reshard_fragment_count.restype = c.c_int64
    L.tc_reshard_fragments.argtypes = [P, c.c_int64, c.c_int32, c.c_int32, P, c.c_int64,
                                       c.POINTER(c.c_int64)]
    L.tc_reshard_cast_item_count.argtypes = [P, c.c_int64, c.c_int32, c.c_int32]
    L.tc_reshard_cast_item_count.restype = c.c_int64
    L.tc_reshard_cast_items.argtypes = [P, P, c.c_int64, c.c_int32, c.c_int32, P, c.c_int64,
                                        c.POINTER(c.c_int64)]
    L.tc_cast_fp8_workspace.argtypes = [c.c_int64]
    L.tc_cast_fp8_workspace.restype = c.c_size_t
    L.tc_cast_fp8_blockscaled.argtypes = [P, P, P, P, c.c_int64, c.c_int32, P, c.c_size_t, P]
    L.tc_cast_fp8_scaled.argtypes = [P, c.c_int64, c.c_float, P, P]
    L.tc_cast_fp8_prepare.argtypes = [P, P, P, c.c_int64, c.c_int32, P, c.c_size_t, c.POINTER(TilePlan), P]
    L.tc_cast_fp8_planned.argtypes = [P, P, P, P, c.c_size_t, c.POINTER(TilePlan), P]
    L.tc_dequant_fp8_prepare.argtypes = [P, P, P, c.c_int64, c.c_int32, P, c.c_size_t, c.POINTER(TilePlan), P]
    L.tc_dequant_fp8_planned.argtypes = [P, P, P, P, c.c_size_t, c.POINTER(TilePlan), P]
    L.tc_ipc_export.argtypes = [P, c.c_size_t, c.POINTER(_IpcHandle)]
    L.tc_ipc_open.argtypes = [c.POINTER(_IpcHandle), c.POINTER(c.c_void_p)]
    L.tc_ipc_close.argtypes = [c.POINTER(_IpcHandle), P]
    L.tc_dequant_fp8_workspace.argtypes = [c.c_int64]
    L.tc_dequant_fp8_workspace.restype = c.c_size_t
    L.tc_cast_fp8_workspace_tiles.argtypes = [P, c.c_int64]
    L.tc_cast_fp8_workspace_tiles.restype = c.c_size_t
    L.tc_dequant_fp8_workspace_tiles.argtypes = [P, c.c_int64]
    L.tc_dequant_fp8_workspace_tiles.restype = c.c_size_t
    L.tc_dequant_fp8_blockscaled.argtypes = [P, P, P, P, c.c_int64, c.c_int32, P, c.c_size_t, P]
    L.tc_stager_create.argtypes = [c.c_size_t, c.c_int32, c.c_int32, c.POINTER(c.c_void_p)]
    L.tc_stager_destroy.argtypes = [P]
    L.tc_stage_h2d.argtypes = [P, P, P, c.c_size_t, c.c_int32, P]
    L.tc_stage_d2h.argtypes = [P, P, P, c.c_size_t, c.c_int32, P]
    L.tc_hydrate_from_host.argtypes = [P, c.POINTER(_BlockPool), P, c.c_int64, P, c.c_int32, P,
                                       c.c_size_t, P]
    L.tc_publish_to_host.argtypes = [P, c.POINTER(_BlockPool), P, c.c_int64, P, c.c_int32, P,
                                     c.c_size_t, P]
    L.tc_status_string.argtypes = [c.c_int]
    L.tc_status_string.restype = c.c_char_p
    L.tc_last_hip_error.restype = c.c_int
    L.tc_set_validate.argtypes = [c.c_int]
    L.tc_get_validate.restype = c.c_int
    for name in ("tc_gather_blocks", "tc_scatter_blocks", "tc_copy_fragments", "tc_plan_fragments",
                 "tc_plan_fragments_async", "tc_plan_status",
                 "tc_copy_planned", "tc_copy_planned_digest", "tc_digest_planned", "tc_tp_fragments", "tc_tp_cast_item", "tc_reshard_fragments", "tc_reshard_cast_items",
                 "tc_cast_fp8_blockscaled", "tc_dequant_fp8_blockscaled",
                 "tc_cast_fp8_prepare", "tc_cast_fp8_planned", "tc_dequant_fp8_prepare",
                 "tc_dequant_fp8_planned", "tc_ipc_export", "tc_ipc_open", "tc_ipc_close",
                 "tc_cast_fp8_scaled", "tc_stager_create", "tc_stager_destroy", "tc_stage_h2d",
                 "tc_stage_d2h", "tc_hydrate_from_host", "tc_publish_to_host"):
        getattr(L, name).restype = c.c_int
    _lib = L
    return L


def _ok(status: int, what: str) -> None:
    if status != TC_OK:
        raise TcError(status, what)


def _dev_ptr(x) -> int:
    """Device address of a torch tensor (must live on a GPU and be contiguous:
    the library addresses it as one flat byte range) or a raw int."""
    if isinstance(x, int):
        return x
    if not x.is_cuda:
        raise ValueError("expected a device tensor")
    if not x.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    return x.data_ptr()


def _stream(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


# ---------------------------------------------------------------------------
# publish / hydrate
# ---------------------------------------------------------------------------

def _ids(ids) -> int:
    """Element count of an id tensor: the library reads int32 ids."""
    if ids.dtype != _torch().int32:
        raise ValueError(f"ids must be an int32 tensor, not {ids.dtype}")
    return ids.numel()


def _pool(regions, num_blocks: int, block_bytes: int, block_stride: int):
    bases = [_dev_ptr(r) for r in regions]
    arr = (ctypes.c_uint64 * len(bases))(*bases)
    pool = _BlockPool(ctypes.cast(arr, ctypes.POINTER(ctypes.c_uint64)), len(bases), num_blocks,
                      block_bytes, block_stride)
    return pool, arr


def tc_gather_blocks(regions, num_blocks: int, block_bytes: int, block_stride: int, ids, out,
                     stream=None) -> None:
    """out[i, r, :block_bytes] = regions[r][ids[i]*stride : +block_bytes] on the device.

    ``regions``: list of device tensors or device addresses (one per layer and
    K|V); ``ids``: device int32 tensor; ``out``: device tensor of
    len(ids) * len(regions) * block_bytes bytes."""
    n = _ids(ids)
    pool, keep = _pool(regions, num_blocks, block_bytes, block_stride)
    if n and _nbytes(out) < n * len(keep) * block_bytes:
        raise ValueError("output buffer too small")
    _ok(load().tc_gather_blocks(ctypes.byref(pool), _dev_ptr(ids) if n else None, n,
                                _dev_ptr(out) if n else None, _stream(stream)), "tc_gather_blocks")


def tc_scatter_blocks(regions, num_blocks: int, block_bytes: int, block_stride: int, ids, inp,
                      stream=None) -> None:
    """regions[r][ids[i]*stride : +block_bytes] = inp[i, r, :] on the device (ids distinct)."""
    n = _ids(ids)
    pool, keep = _pool(regions, num_blocks, block_bytes, block_stride)
    if n and _nbytes(inp) < n * len(keep) * block_bytes:
        raise ValueError("input buffer too small")
    _ok(load().tc_scatter_blocks(ctypes.byref(pool), _dev_ptr(ids) if n else None, n,
                                 _dev_ptr(inp) if n else None, _stream(stream)), "tc_scatter_blocks")


# ---------------------------------------------------------------------------
# fragments
# ---------------------------------------------------------------------------

def tc_copy_fragments_workspace(n: int) -> int:
    return int(load().tc_copy_fragments_workspace(int(n)))


def tc_copy_fragments_workspace_min(n: int) -> int:
    return int(load().tc_copy_fragments_workspace_min(int(n)))


def _frag_count(frags) -> int:
    if frags.dtype not in (_torch().uint64, _torch().int64):
        raise ValueError(f"fragments must be a uint64/int64 tensor, not {frags.dtype}")
    nb = _nbytes(frags)
    if nb % 24:
        raise ValueError("fragment tensor is not a whole number of (src_off, dst_off, len) rows")
    return nb // 24


def tc_copy_fragments(src, dst, frags, workspace, stream=None) -> None:
    """Copy every (src_off, dst_off, len) row of the device tensor ``frags``
    (uint64/int64, shape [n, 3]) from ``src`` to ``dst``.  Asynchronous: the
    plan and the copy are enqueued on ``stream``; failures the plan finds on
    the device are reported by ``tc_plan_status(workspace)``."""
    n = _frag_count(frags)
    _ok(load().tc_copy_fragments(_dev_ptr(src), _dev_ptr(dst), _dev_ptr(frags) if n else None, n,
                                 _dev_ptr(workspace), _nbytes(workspace), _stream(stream)),
        "tc_copy_fragments")


def tc_plan_fragments(frags, workspace, stream=None) -> int:
    """Plan the copy of ``frags`` into ``workspace``; returns the task count."""
    n = _frag_count(frags)
    total = ctypes.c_uint64(0)
    _ok(load().tc_plan_fragments(_dev_ptr(frags) if n else None, n, _dev_ptr(workspace),
                                 _nbytes(workspace), ctypes.byref(total), _stream(stream)),
        "tc_plan_fragments")
    return int(total.value)


def tc_plan_fragments_async(frags, workspace, stream=None) -> None:
    """Enqueue the plan of ``frags`` into ``workspace`` without waiting for it."""
    n = _frag_count(frags)
    _ok(load().tc_plan_fragments_async(_dev_ptr(frags) if n else None, n, _dev_ptr(workspace),
                                       _nbytes(workspace), _stream(stream)),
        "tc_plan_fragments_async")


def tc_plan_status(workspace, stream=None) -> int:
    """Wait for the plan in ``workspace`` and return its task count; raises
    TcError with the plan's status if the plan failed on the device."""
    total = ctypes.c_uint64(0)
    _ok(load().tc_plan_status(_dev_ptr(workspace), _nbytes(workspace), ctypes.byref(total),
                              _stream(stream)), "tc_plan_status")
    return int(total.value)


def tc_copy_planned(src, dst, workspace, total_tasks=None, stream=None) -> None:
    """Copy with a plan made by tc_plan_fragments (same workspace, unchanged).
    ``total_tasks=None`` lets the kernel read the plan's count on the device."""
    total = TASKS_FROM_PLAN if total_tasks is None else int(total_tasks)
    _ok(load().tc_copy_planned(_dev_ptr(src), _dev_ptr(dst), _dev_ptr(workspace),
                               _nbytes(workspace), total, _stream(stream)),
        "tc_copy_planned")


def _digest_out(digests, n: int) -> int:
    if digests.dtype not in (_torch().uint64, _torch().int64) or digests.numel() < 2 * n:
        raise ValueError("digests must be a device uint64/int64 tensor of at least 2n words")
    return _dev_ptr(digests)


def _torch():
    import torch
    return torch


def tc_copy_planned_digest(src, dst, workspace, total_tasks: int, n: int, digests,
                           stream=None) -> None:
    """tc_copy_planned that also writes digests[f] = (S1, S2) of each of the
    plan's n fragments (``digests``: device uint64/int64 tensor, 2n words)."""
    _ok(load().tc_copy_planned_digest(_dev_ptr(src), _dev_ptr(dst), _dev_ptr(workspace),
                                      _nbytes(workspace), int(total_tasks), int(n),
                                      _digest_out(digests, n), _stream(stream)),
        "tc_copy_planned_digest")


def tc_digest_planned(base, side: int, workspace, total_tasks: int, n: int, digests,
                      stream=None) -> None:
    """Digests of the plan's fragments read from ``base`` at their source
    (DIGEST_SRC) or destination (DIGEST_DST) offsets."""
    _ok(load().tc_digest_planned(_dev_ptr(base), int(side), _dev_ptr(workspace),
                                 _nbytes(workspace), int(total_tasks), int(n),
                                 _digest_out(digests, n), _stream(stream)),
        "tc_digest_planned")


# ---------------------------------------------------------------------------
# host <-> device staging
# ---------------------------------------------------------------------------

def _host(buf):
    """(address, bytes, pinned) of a host buffer: a numpy array (pageable) or
    a CPU torch tensor (pinned when it was allocated with pin_memory)."""
    if isinstance(buf, np.ndarray):
        if not buf.flags["C_CONTIGUOUS"]:
            raise ValueError("host buffer must be contiguous")
        return buf.ctypes.data, buf.nbytes, False
    if buf.is_cuda:
        raise ValueError("expected a host buffer")
    if not buf.is_contiguous():
        raise ValueError("host buffer must be contiguous")
    return buf.data_ptr(), _nbytes(buf), bool(buf.is_pinned())


def _flags(pinned_detected: bool, pinned) -> int:
    use = pinned_detected if pinned is None else bool(pinned)
    return HOST_PINNED if use else 0


def tc_stager_create(slot_bytes: int = 0, slots: int = 0, host_threads: int = 0) -> int:
    """A stager bound to the current device; returns its handle."""
    h = ctypes.c_void_p(0)
    _ok(load().tc_stager_create(int(slot_bytes), int(slots), int(host_threads), ctypes.byref(h)),
        "tc_stager_create")
    return int(h.value)


def tc_stager_destroy(stager: int) -> None:
    _ok(load().tc_stager_destroy(stager), "tc_stager_destroy")


def tc_stage_h2d(stager: int, host_src, dev_dst, nbytes=None, pinned=None, stream=None) -> None:
    """Copy host bytes to the device through the pinned ring (or directly if pinned)."""
    a, n, det = _host(host_src)
    n = n if nbytes is None else int(nbytes)
    if n > _nbytes(dev_dst):
        raise ValueError("device buffer too small")
    _ok(load().tc_stage_h2d(stager, a, _dev_ptr(dev_dst), n, _flags(det, pinned), _stream(stream)),
        "tc_stage_h2d")


def tc_stage_d2h(stager: int, dev_src, host_dst, nbytes=None, pinned=None, stream=None) -> None:
    """Copy device bytes into host memory; returns when host_dst holds them."""
    a, n, det = _host(host_dst)
    n = n if nbytes is None else int(nbytes)
    if n > _nbytes(dev_src):
        raise ValueError("device buffer too small")
    _ok(load().tc_stage_d2h(stager, _dev_ptr(dev_src), a, n, _flags(det, pinned), _stream(stream)),
        "tc_stage_d2h")


def tc_hydrate_from_host(stager: int, regions, num_blocks: int, block_bytes: int, block_stride: int,
                         ids, host_src, dev_stage, pinned=None, stream=None) -> None:
    """Scatter a host-resident transfer buffer (layout of tc_gather_blocks)
    into the device block pool, staged through ``dev_stage``."""
    n = _ids(ids)
    pool, keep = _pool(regions, num_blocks, block_bytes, block_stride)
    a, hb, det = _host(host_src)
    if n and hb < n * len(keep) * block_bytes:
        raise ValueError("host buffer too small")
    _ok(load().tc_hydrate_from_host(stager, ctypes.byref(pool), _dev_ptr(ids) if n else None, n, a,
                                    _flags(det, pinned), _dev_ptr(dev_stage), _nbytes(dev_stage),
                                    _stream(stream)), "tc_hydrate_from_host")


def tc_publish_to_host(stager: int, regions, num_blocks: int, block_bytes: int, block_stride: int,
                       ids, host_dst, dev_stage, pinned=None, stream=None) -> None:
    """Gather the pool's blocks of ``ids`` into host memory (blocks until done)."""
    n = _ids(ids)
    pool, keep = _pool(regions, num_blocks, block_bytes, block_stride)
    a, hb, det = _host(host_dst)
    if n and hb < n * len(keep) * block_bytes:
        raise ValueError("host buffer too small")
    _ok(load().tc_publish_to_host(stager, ctypes.byref(pool), _dev_ptr(ids) if n else None, n, a,
                                  _flags(det, pinned), _dev_ptr(dev_stage), _nbytes(dev_stage),
                                  _stream(stream)), "tc_publish_to_host")


class Stager:
    """Owns a stager handle (``with Stager() as st: ...``)."""

    def __init__(self, slot_bytes: int = 0, slots: int = 0, host_threads: int = 0):
        self.handle = tc_stager_create(slot_bytes, slots, host_threads)

    def close(self) -> None:
        if self.handle:
            tc_stager_destroy(self.handle)
            self.handle = 0

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        # at interpreter shutdown the HIP runtime may already be gone: leave
        # the stager to the process exit then
        if not self.handle or _sys.is_finalizing():
            return
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------------------
# tensor-parallel views (host builders)
# ---------------------------------------------------------------------------

def _views(views) -> np.ndarray:
    v = np.ascontiguousarray(views, dtype=TP_VIEW_DTYPE).reshape(-1)
    return v


def tc_tp_fragment_count(views, tp: int, rank: int) -> int:
    v = _views(views)
    n = int(load().tc_tp_fragment_count(v.ctypes.data if v.size else None, v.size, tp, rank))
    if n < 0:
        raise TcError(1, "tc_tp_fragment_count")
    return n


def tc_tp_fragments(views, tp: int, rank: int) -> np.ndarray:
    """Fragments (uint64 [m, 3]) that copy rank ``rank``'s slices."""
    v = _views(views)
    m = tc_tp_fragment_count(v, tp, rank)
    out = np.zeros((m, 3), dtype=np.uint64)
    written = ctypes.c_int64(0)
    _ok(load().tc_tp_fragments(v.ctypes.data if v.size else None, v.size, tp, rank,
                               out.ctypes.data if m else None, m, ctypes.byref(written)),
        "tc_tp_fragments")
    return out[:written.value]


def tc_tp_cast_item(view, tp: int, rank: int, scale_off: int) -> np.ndarray:
    """The cast item (CAST_ITEM_DTYPE record) for a rank's slice of a bf16 weight."""
    v = _views([view] if np.ndim(view) == 0 else view)
    assert v.size == 1
    out = np.zeros(1, dtype=CAST_ITEM_DTYPE)
    _ok(load().tc_tp_cast_item(v.ctypes.data, tp, rank, scale_off, out.ctypes.data),
        "tc_tp_cast_item")
    return out[0]


def _reshard_array(views):
    """views: sequence of (src_offsets, rows, cols, elem_bytes, split, dst_off)."""
    keep = []
    arr = (_ReshardView * len(views))()
    for k, (offs, rows, cols, eb, split, dst_off) in enumerate(views):
        o = (ctypes.c_uint64 * len(offs))(*[int(x) for x in offs])
        keep.append(o)
        arr[k] = _ReshardView(ctypes.cast(o, ctypes.POINTER(ctypes.c_uint64)), rows, cols, eb, split,
                              len(offs), 0, dst_off)
    return arr, keep


def tc_reshard_fragment_count(views, dst_tp: int, dst_rank: int) -> int:
    arr, _keep = _reshard_array(views)
    n = int(load().tc_reshard_fragment_count(arr if len(views) else None, len(views), dst_tp, dst_rank))
    if n < 0:
        raise TcError(1, "tc_reshard_fragment_count")
    return n


def tc_reshard_fragments(views, dst_tp: int, dst_rank: int) -> np.ndarray:
    """Fragments (uint64 [m, 3]) that build rank ``dst_rank`` of a ``dst_tp``-way
    split from the source slices described by ``views``."""
    arr, _keep = _reshard_array(views)
    m = tc_reshard_fragment_count(views, dst_tp, dst_rank)
    out = np.zeros((m, 3), dtype=np.uint64)
    written = ctypes.c_int64(0)
    _ok(load().tc_reshard_fragments(arr if len(views) else None, len(views), dst_tp, dst_rank,
                                    out.ctypes.data if m else None, m, ctypes.byref(written)),
        "tc_reshard_fragments")
    return out[:written.value]


def tc_reshard_cast_item_count(views, dst_tp: int, dst_rank: int) -> int:
    arr, _keep = _reshard_array(views)
    n = int(load().tc_reshard_cast_item_count(arr if len(views) else None, len(views), dst_tp, dst_rank))
    if n < 0:
        raise TcError(1, "tc_reshard_cast_item_count")
    return n


def tc_reshard_cast_items(views, scale_off, dst_tp: int, dst_rank: int) -> np.ndarray:
    """CAST_ITEM_DTYPE records that cast rank ``dst_rank``'s slices of a
    ``dst_tp``-way split straight from the bf16 source slices of ``views``
    (byte offsets; fp8 destination offsets) into fp8 with per-view scale
    grids at ``scale_off`` (floats)."""
    arr, _keep = _reshard_array(views)
    so = np.ascontiguousarray(scale_off, dtype=np.uint64).reshape(-1)
    if so.size != len(views):
        raise ValueError("one scale offset per view")
    m = tc_reshard_cast_item_count(views, dst_tp, dst_rank)
    out = np.zeros(m, dtype=CAST_ITEM_DTYPE)
    written = ctypes.c_int64(0)
    _ok(load().tc_reshard_cast_items(arr if len(views) else None, so.ctypes.data if so.size else None,
                                     len(views), dst_tp, dst_rank, out.ctypes.data if m else None, m,
                                     ctypes.byref(written)), "tc_reshard_cast_items")
    return out[:written.value]


# ---------------------------------------------------------------------------
# transform_into: fp8 cast
# ---------------------------------------------------------------------------

def tc_cast_fp8_workspace(n_items: int) -> int:
    return int(load().tc_cast_fp8_workspace(int(n_items)))


def tc_cast_fp8_workspace_tiles(items) -> int:
    """Workspace bytes with room for the per-tile table of ``items`` (host
    CAST_ITEM_DTYPE records); 0 for an invalid item."""
    it = np.ascontiguousarray(items, dtype=CAST_ITEM_DTYPE).reshape(-1)
    return int(load().tc_cast_fp8_workspace_tiles(it.ctypes.data if it.size else None, it.size))


def tc_cast_fp8_blockscaled(src, dst, scales, items, workspace, stream=None, tile: int = 128) -> None:
    """Cast every item; ``items`` is a host numpy array of CAST_ITEM_DTYPE
    records, written into ``workspace`` on the stream by kernels that carry
    it in their arguments (the array may be reused once the call returns).
    A workspace of tc_cast_fp8_workspace_tiles(items) bytes also holds the
    per-tile table, which the cast then reads."""
    it = np.ascontiguousarray(items, dtype=CAST_ITEM_DTYPE).reshape(-1)
    n = it.size
    _ok(load().tc_cast_fp8_blockscaled(_dev_ptr(src), _dev_ptr(dst), _dev_ptr(scales),
                                       it.ctypes.data if n else None, n, tile, _dev_ptr(workspace),
                                       _nbytes(workspace), _stream(stream)),
        "tc_cast_fp8_blockscaled")


def tc_cast_fp8_prepare(src, dst, items, workspace, stream=None, tile: int = 128) -> TilePlan:
    """Write the cast's tile table for ``items`` into ``workspace``; returns
    the plan for tc_cast_fp8_planned (bases with the same alignment)."""
    it = np.ascontiguousarray(items, dtype=CAST_ITEM_DTYPE).reshape(-1)
    n = it.size
    plan = TilePlan()
    _ok(load().tc_cast_fp8_prepare(_dev_ptr(src), _dev_ptr(dst), it.ctypes.data if n else None, n, tile,
                                   _dev_ptr(workspace), _nbytes(workspace), ctypes.byref(plan),
                                   _stream(stream)), "tc_cast_fp8_prepare")
    return plan


def tc_cast_fp8_planned(src, dst, scales, workspace, plan: TilePlan, stream=None) -> None:
    """Launch only the cast kernels, with a table prepared in ``workspace``."""
    _ok(load().tc_cast_fp8_planned(_dev_ptr(src), _dev_ptr(dst), _dev_ptr(scales), _dev_ptr(workspace),
                                   _nbytes(workspace), ctypes.byref(plan), _stream(stream)),
        "tc_cast_fp8_planned")


def tc_cast_fp8_scaled(src, scale: float, dst, stream=None) -> None:
    """dst[i] = E4M3(RN_f32(src[i] / scale)) for a bf16 device tensor ``src``."""
    if src.element_size() != 2:
        raise ValueError("src must hold bf16 (2-byte) elements")
    n = src.numel()
    if _nbytes(dst) < n:
        raise ValueError("dst too small: one byte per element")
    _ok(load().tc_cast_fp8_scaled(_dev_ptr(src) if n else None, n, float(scale),
                                  _dev_ptr(dst) if n else None, _stream(stream)),
        "tc_cast_fp8_scaled")


def tc_dequant_fp8_workspace(n_items: int) -> int:
    return int(load().tc_dequant_fp8_workspace(int(n_items)))


def tc_dequant_fp8_workspace_tiles(items) -> int:
    """Workspace bytes with room for the per-tile table of ``items`` (host
    DEQUANT_ITEM_DTYPE records); 0 for an invalid item."""
    it = np.ascontiguousarray(items, dtype=DEQUANT_ITEM_DTYPE).reshape(-1)
    return int(load().tc_dequant_fp8_workspace_tiles(it.ctypes.data if it.size else None, it.size))


def tc_dequant_fp8_blockscaled(codes, scales, dst, items, workspace, stream=None, tile: int = 128) -> None:
    """bf16 = RN_bf16(RN_f32(E4M3(q) * s)) for every item; ``items`` is a host
    numpy array of DEQUANT_ITEM_DTYPE records."""
    it = np.ascontiguousarray(items, dtype=DEQUANT_ITEM_DTYPE).reshape(-1)
    n = it.size
    _ok(load().tc_dequant_fp8_blockscaled(_dev_ptr(codes), _dev_ptr(scales), _dev_ptr(dst),
                                          it.ctypes.data if n else None, n, tile,
                                          _dev_ptr(workspace), _nbytes(workspace), _stream(stream)),
        "tc_dequant_fp8_blockscaled")


def tc_dequant_fp8_prepare(codes, dst, items, workspace, stream=None, tile: int = 128) -> TilePlan:
    """Write the inverse cast's tile table into ``workspace``; returns its plan."""
    it = np.ascontiguousarray(items, dtype=DEQUANT_ITEM_DTYPE).reshape(-1)
    n = it.size
    plan = TilePlan()
    _ok(load().tc_dequant_fp8_prepare(_dev_ptr(codes), _dev_ptr(dst), it.ctypes.data if n else None, n,
                                      tile, _dev_ptr(workspace), _nbytes(workspace), ctypes.byref(plan),
                                      _stream(stream)), "tc_dequant_fp8_prepare")
    return plan


def tc_dequant_fp8_planned(codes, scales, dst, workspace, plan: TilePlan, stream=None) -> None:
    """Launch only the inverse-cast kernels, with a prepared table."""
    _ok(load().tc_dequant_fp8_planned(_dev_ptr(codes), _dev_ptr(scales), _dev_ptr(dst),
                                      _dev_ptr(workspace), _nbytes(workspace), ctypes.byref(plan),
                                      _stream(stream)), "tc_dequant_fp8_planned")


# ---------------------------------------------------------------------------
# zero-copy sharing between processes (HIP IPC)
# ---------------------------------------------------------------------------

def tc_ipc_export(dev, nbytes=None) -> bytes:
    """Handle (plain bytes) for a device tensor's bytes, or ``nbytes`` bytes at
    a device address; send it to another process on this host."""
    n = _nbytes(dev) if nbytes is None else int(nbytes)
    h = _IpcHandle()
    _ok(load().tc_ipc_export(_dev_ptr(dev), n, ctypes.byref(h)), "tc_ipc_export")
    return bytes(h)


def _ipc_handle(handle: bytes) -> _IpcHandle:
    if len(handle) != IPC_HANDLE_BYTES:
        raise ValueError(f"an IPC handle has {IPC_HANDLE_BYTES} bytes")
    return _IpcHandle.from_buffer_copy(handle)


def tc_ipc_open(handle: bytes) -> int:
    """Map an exported range into this process; returns its device address."""
    h = _ipc_handle(handle)
    p = ctypes.c_void_p(0)
    _ok(load().tc_ipc_open(ctypes.byref(h), ctypes.byref(p)), "tc_ipc_open")
    return int(p.value)


def tc_ipc_close(handle: bytes, dev_ptr: int) -> None:
    h = _ipc_handle(handle)
    _ok(load().tc_ipc_close(ctypes.byref(h), ctypes.c_void_p(dev_ptr)), "tc_ipc_close")


# ---------------------------------------------------------------------------

def tc_status_string(status: int) -> str:
    return load().tc_status_string(int(status)).decode()


def tc_last_hip_error() -> int:
    return int(load().tc_last_hip_error())


def tc_set_validate(on: bool) -> None:
    load().tc_set_validate(1 if on else 0)


def tc_get_validate() -> bool:
    return bool(load().tc_get_validate())
