"""CPU oracle for the tensor-lifecycle data path.

TEST INFRASTRUCTURE ONLY: tests, the smoke check and the benchmark's CPU
baseline may import this package; the product library never does.  It
shares no code with the GPU path: the byte movers and the E4M3 cast live in
``oracle.c`` (loaded through ctypes), and the tensor-parallel slicing is
written here with plain numpy indexing.

What each function follows:

* ``gather_blocks`` / ``scatter_blocks`` -- publish (export a request's KV
  blocks from the engine into one contiguous buffer) and hydrate (load them
  back into engine blocks), paper Sec. 3.2 "Operation", Table 2.
* ``copy_fragments`` -- batched replica moves (prefetch_many, Table 2) and
  the transfer stage of the materialization pipeline (Sec. 5).
* ``tp_shard`` -- Artifact.view(slice) + tensor_dict(): each tensor-parallel
  rank materializes only its slice of every weight (Sec. 6.1 and 6.2).
* ``cast_fp8_blockscaled`` / ``cast_fp8_scaled`` / ``e4m3_encode`` -- one
  concrete transform_into `spec` rule (Table 2): bf16 -> OCP FP8 E4M3 with
  an fp32 scale per 128x128 tile.
* ``fragment_digests`` -- a per-fragment integrity digest, for the verify
  stage of the materialization pipeline (Sec. 5).
* ``dequant_fp8_blockscaled`` -- its inverse, back to bf16, for resharding
  stored fp8 checkpoints into other layouts (Sec. 2.1, Sec. 7).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# TC_ORACLE_LIB loads another build of oracle.c instead (the mutation test
# runs the pins against deliberately broken copies that way).
_LIB_PATH = os.environ.get("TC_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

TILE = 128
E4M3_MAX = 448.0


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        if os.environ.get("TC_ORACLE_LIB"):
            raise RuntimeError(f"TC_ORACLE_LIB names a missing library: {_LIB_PATH}")
        from . import build as _build
        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    c = ctypes
    lib.orc_threads.restype = c.c_int
    lib.orc_set_threads.argtypes = [c.c_int]
    lib.orc_gather_blocks.argtypes = [c.POINTER(c.c_void_p), c.c_int32, c.c_int64,
                                      c.c_int64, c.c_int64, c.c_void_p, c.c_int64, c.c_void_p]
    lib.orc_gather_blocks.restype = c.c_int
    lib.orc_scatter_blocks.argtypes = lib.orc_gather_blocks.argtypes
    lib.orc_scatter_blocks.restype = c.c_int
    lib.orc_copy_fragments.argtypes = [c.c_void_p, c.c_void_p, c.c_void_p, c.c_int64]
    lib.orc_copy_fragments.restype = None
    lib.orc_e4m3_encode.argtypes = [c.c_float]
    lib.orc_e4m3_encode.restype = c.c_uint8
    lib.orc_e4m3_decode.argtypes = [c.c_uint8]
    lib.orc_e4m3_decode.restype = c.c_float
    lib.orc_cast_fp8_scaled.argtypes = [c.c_void_p, c.c_int64, c.c_float, c.c_void_p]
    lib.orc_cast_fp8_scaled.restype = None
    lib.orc_cast_fp8_blockscaled.argtypes = [c.c_void_p, c.c_int64, c.c_int64, c.c_int64,
                                             c.c_void_p, c.c_int64, c.c_void_p, c.c_int64]
    lib.orc_cast_fp8_blockscaled.restype = None
    lib.orc_dequant_fp8_blockscaled.argtypes = [c.c_void_p, c.c_int64, c.c_int64, c.c_int64,
                                                c.c_void_p, c.c_int64, c.c_void_p, c.c_int64]
    lib.orc_dequant_fp8_blockscaled.restype = None
    lib.orc_fragment_digests.argtypes = [c.c_void_p, c.c_void_p, c.c_int64, c.c_int, c.c_void_p]
    lib.orc_fragment_digests.restype = None
    lib.orc_bf16_round.argtypes = [c.c_float]
    lib.orc_bf16_round.restype = c.c_uint16
    _lib = lib
    return lib


def threads() -> int:
    return _load().orc_threads()


def set_threads(n: int) -> None:
    _load().orc_set_threads(int(n))


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


# ---------------------------------------------------------------------------
# publish / hydrate
# ---------------------------------------------------------------------------

def gather_blocks(regions, block_bytes: int, block_stride: int, ids: np.ndarray) -> np.ndarray:
    """Export: out[i, r, :] = regions[r][ids[i]*stride : ids[i]*stride + B].

    ``regions`` is a list of 1-D uint8 arrays (one per layer and K/V)."""
    lib = _load()
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    R = len(regions)
    nb = min(_num_blocks(r, block_bytes, block_stride) for r in regions)
    out = np.empty((len(ids), R, block_bytes), dtype=np.uint8)
    ptrs = (ctypes.c_void_p * R)(*[_ptr(r) for r in regions])
    rc = lib.orc_gather_blocks(ptrs, R, nb, block_bytes, block_stride, _ptr(ids), len(ids), _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle gather: bad ids (code {rc})")
    return out


def scatter_blocks(regions, block_bytes: int, block_stride: int, ids: np.ndarray,
                   data: np.ndarray) -> None:
    """Import: regions[r][ids[i]*stride : +B] = data[i, r, :] (ids distinct)."""
    lib = _load()
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    data = np.ascontiguousarray(data, dtype=np.uint8)
    R = len(regions)
    assert data.size == len(ids) * R * block_bytes
    nb = min(_num_blocks(r, block_bytes, block_stride) for r in regions)
    ptrs = (ctypes.c_void_p * R)(*[_ptr(r) for r in regions])
    rc = lib.orc_scatter_blocks(ptrs, R, nb, block_bytes, block_stride, _ptr(ids), len(ids), _ptr(data))
    if rc != 0:
        raise ValueError(f"oracle scatter: bad ids (code {rc})")


def _num_blocks(region: np.ndarray, block_bytes: int, block_stride: int) -> int:
    if region.size < block_bytes:
        return 0
    return (region.size - block_bytes) // block_stride + 1


# ---------------------------------------------------------------------------
# prefetch_many / transfer stage
# ---------------------------------------------------------------------------

def copy_fragments(src: np.ndarray, dst: np.ndarray, frags: np.ndarray) -> None:
    """dst[d_off : d_off+len] = src[s_off : s_off+len] for each (s_off, d_off, len) row."""
    frags = np.ascontiguousarray(frags, dtype=np.uint64).reshape(-1, 3)
    if len(frags):
        ends_s = frags[:, 0] + frags[:, 2]
        ends_d = frags[:, 1] + frags[:, 2]
        if int(ends_s.max()) > src.size or int(ends_d.max()) > dst.size:
            raise ValueError("oracle copy: fragment out of range")
    _load().orc_copy_fragments(_ptr(src), _ptr(dst), _ptr(frags), len(frags))


# ---------------------------------------------------------------------------
# view(slice) + tensor_dict(): tensor-parallel shard materialization
# ---------------------------------------------------------------------------

def tp_slice(w: np.ndarray, split: str, tp: int, rank: int) -> np.ndarray:
    """The rank's slice of a 2-D weight.  ``split`` 'rows' keeps rows
    [rank*R/tp, (rank+1)*R/tp) (column-parallel layers), 'cols' keeps that
    range of columns (row-parallel layers), 'none' keeps the whole matrix."""
    rows, cols = w.shape
    if split == "rows":
        assert rows % tp == 0
        k = rows // tp
        return w[rank * k:(rank + 1) * k, :]
    if split == "cols":
        assert cols % tp == 0
        k = cols // tp
        return w[:, rank * k:(rank + 1) * k]
    if split == "none":
        return w
    raise ValueError(split)


def tp_shard(stream: np.ndarray, spec, tp: int, rank: int) -> np.ndarray:
    """Walk a contiguous stream of row-major matrices (in ``spec`` order) and
    concatenate the rank's slices, each written densely row-major.

    ``stream`` is a 1-D array of elements; ``spec`` is a sequence of
    (name, rows, cols, split)."""
    parts = []
    off = 0
    for (_name, rows, cols, split) in spec:
        w = stream[off:off + rows * cols].reshape(rows, cols)
        off += rows * cols
        parts.append(np.ascontiguousarray(tp_slice(w, split, tp, rank)).reshape(-1))
    assert off == stream.size, "spec does not cover the stream"
    return np.concatenate(parts) if parts else stream[:0].copy()


# ---------------------------------------------------------------------------
# transform_into with an fp8 spec
# ---------------------------------------------------------------------------

def e4m3_encode(v: float) -> int:
    return int(_load().orc_e4m3_encode(float(v)))


def e4m3_decode(code: int) -> float:
    return float(_load().orc_e4m3_decode(int(code)))


def cast_fp8_scaled(x_bits: np.ndarray, scale: float) -> np.ndarray:
    """Codes of RN_f32(bf16(x) / scale); ``x_bits`` are raw bf16 bit patterns."""
    x = np.ascontiguousarray(x_bits, dtype=np.uint16).reshape(-1)
    q = np.empty(x.size, dtype=np.uint8)
    _load().orc_cast_fp8_scaled(_ptr(x), x.size, float(np.float32(scale)), _ptr(q))
    return q.reshape(np.shape(x_bits))


def scale_grid(rows: int, cols: int):
    return (rows + TILE - 1) // TILE, (cols + TILE - 1) // TILE


def cast_fp8_blockscaled(x_bits: np.ndarray):
    """Cast one 2-D bf16 matrix (raw bit patterns, any row stride) to E4M3
    codes [rows, cols] and fp32 scales [ceil(rows/128), ceil(cols/128)]."""
    x = np.asarray(x_bits)
    assert x.dtype == np.uint16 and x.ndim == 2
    if x.strides[1] != 2:
        x = np.ascontiguousarray(x)
    rows, cols = x.shape
    ld = x.strides[0] // 2
    q = np.empty((rows, cols), dtype=np.uint8)
    tr, tc = scale_grid(rows, cols)
    s = np.empty((tr, tc), dtype=np.float32)
    if rows and cols:
        _load().orc_cast_fp8_blockscaled(_ptr(x), rows, cols, ld, _ptr(q), cols, _ptr(s), tc)
    return q, s


def bf16_round(v: float) -> int:
    return int(_load().orc_bf16_round(float(v)))


def dequant_fp8_blockscaled(q: np.ndarray, scales: np.ndarray) -> np.ndarray:
    """bf16 bit patterns [rows, cols] of RN_bf16(RN_f32(dec(q) * s)) with s the
    scale of each element's 128x128 tile."""
    q = np.asarray(q)
    assert q.dtype == np.uint8 and q.ndim == 2
    if q.strides[1] != 1:
        q = np.ascontiguousarray(q)
    rows, cols = q.shape
    s = np.ascontiguousarray(scales, dtype=np.float32)
    assert s.shape == scale_grid(rows, cols)
    y = np.empty((rows, cols), dtype=np.uint16)
    if rows and cols:
        _load().orc_dequant_fp8_blockscaled(_ptr(q), rows, cols, q.strides[0], _ptr(s), s.shape[1],
                                            _ptr(y), cols)
    return y


def fragment_digests(buf: np.ndarray, frags: np.ndarray, use_src: bool = True) -> np.ndarray:
    """[n, 2] uint64: S1 = sum of the fragment's bytes, S2 = sum of (i+1)*b_i,
    both mod 2^64, over the bytes at src_off (or dst_off) of each fragment."""
    frags = np.ascontiguousarray(frags, dtype=np.uint64).reshape(-1, 3)
    col = 0 if use_src else 1
    if len(frags) and int((frags[:, col] + frags[:, 2]).max()) > buf.size:
        raise ValueError("oracle digest: fragment out of range")
    out = np.zeros((len(frags), 2), dtype=np.uint64)
    _load().orc_fragment_digests(_ptr(buf), _ptr(frags), len(frags), 1 if use_src else 0, _ptr(out))
    return out
