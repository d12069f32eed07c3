"""Describe a model's weights as tensor-parallel views.

The source is one contiguous stream of row-major matrices in spec order
(each (name, rows, cols, split) entry directly follows the previous one);
the destination is the rank's shard: its slices in the same order, each
packed densely row-major.  These helpers only compute the offsets of that
layout; the moves themselves are described by the library's builders
(``tc_tp_fragments``, ``tc_tp_cast_item``) and done by its kernels.
"""
from __future__ import annotations

import numpy as np

from . import (CAST_ITEM_DTYPE, DEQUANT_ITEM_DTYPE, SPLIT_COLS, SPLIT_NONE, SPLIT_ROWS,
               TP_VIEW_DTYPE, tc_tp_cast_item)

_SPLIT = {"rows": SPLIT_ROWS, "cols": SPLIT_COLS, "none": SPLIT_NONE}


def slice_shape(rows: int, cols: int, split: str, tp: int):
    if split == "rows":
        return rows // tp, cols
    if split == "cols":
        return rows, cols // tp
    return rows, cols


def stream_views(spec, tp: int, elem_bytes: int = 2, dst_elem_bytes: int | None = None) -> np.ndarray:
    """One TP_VIEW_DTYPE record per matrix.  ``dst_elem_bytes`` sets the size
    of a destination element used for dst offsets (defaults to elem_bytes;
    1 for an fp8 destination)."""
    deb = elem_bytes if dst_elem_bytes is None else dst_elem_bytes
    v = np.zeros(len(spec), dtype=TP_VIEW_DTYPE)
    src = dst = 0
    for k, (_name, rows, cols, split) in enumerate(spec):
        sr, sc = slice_shape(rows, cols, split, tp)
        v[k] = (src, rows, cols, cols, dst, sc, elem_bytes, _SPLIT[split])
        src += rows * cols * elem_bytes
        dst += sr * sc * deb
    return v


def shard_elems(spec, tp: int) -> int:
    total = 0
    for (_name, rows, cols, split) in spec:
        sr, sc = slice_shape(rows, cols, split, tp)
        total += sr * sc
    return total


def scale_elems(spec, tp: int, tile: int = 128) -> int:
    total = 0
    for (_name, rows, cols, split) in spec:
        sr, sc = slice_shape(rows, cols, split, tp)
        total += ((sr + tile - 1) // tile) * ((sc + tile - 1) // tile)
    return total


def cast_items(spec, tp: int, rank: int) -> np.ndarray:
    """CAST_ITEM_DTYPE records that cast rank ``rank``'s bf16 slices of a
    contiguous bf16 stream into a packed fp8 shard with packed scale grids."""
    views = stream_views(spec, tp, elem_bytes=2, dst_elem_bytes=1)
    items = np.zeros(len(spec), dtype=CAST_ITEM_DTYPE)
    scale_off = 0
    for k, (_name, rows, cols, split) in enumerate(spec):
        items[k] = tc_tp_cast_item(views[k], tp, rank, scale_off)
        sr, sc = slice_shape(rows, cols, split, tp)
        scale_off += ((sr + 127) // 128) * ((sc + 127) // 128)
    return items


def shard_slice_offsets(spec, tp: int, elem_bytes: int = 2):
    """Byte offset of every matrix's slice inside one rank's packed shard (spec
    order), and the shard's size in bytes."""
    offs = []
    off = 0
    for (_name, rows, cols, split) in spec:
        sr, sc = slice_shape(rows, cols, split, tp)
        offs.append(off)
        off += sr * sc * elem_bytes
    return offs, off


def reshard_views(spec, src_tp: int, dst_tp: int, elem_bytes: int = 2, dst_elem_bytes: int | None = None):
    """Views for tc_reshard_fragments: the source buffer holds the src_tp
    shards one after another (rank-major, each packed in spec order); the
    destination is one rank's packed shard of the dst_tp split
    (``dst_elem_bytes`` per element there; 1 for an fp8 destination)."""
    soffs, sbytes = shard_slice_offsets(spec, src_tp, elem_bytes)
    doffs, _ = shard_slice_offsets(spec, dst_tp, elem_bytes if dst_elem_bytes is None else dst_elem_bytes)
    out = []
    for k, (_name, rows, cols, split) in enumerate(spec):
        src = [r * sbytes + soffs[k] for r in range(src_tp)]
        out.append((src, rows, cols, elem_bytes, _SPLIT[split], doffs[k]))
    return out


def dequant_items(spec, tp: int):
    """DEQUANT_ITEM_DTYPE records that turn one rank's packed fp8 shard (codes
    and scale grids laid out as cast_items writes them) back into its packed
    bf16 shard."""
    items = np.zeros(len(spec), dtype=DEQUANT_ITEM_DTYPE)
    q_off = s_off = 0
    for k, (_name, rows, cols, split) in enumerate(spec):
        sr, sc = slice_shape(rows, cols, split, tp)
        tcn = (sc + 127) // 128
        items[k] = (q_off, sr, sc, sc, q_off, sc, s_off, tcn)
        q_off += sr * sc
        s_off += ((sr + 127) // 128) * tcn
    return items


def scale_offsets(spec, tp: int, tile: int = 128):
    """Float offset of every matrix's scale grid inside one rank's packed
    scale buffer (spec order)."""
    offs = []
    off = 0
    for (_name, rows, cols, split) in spec:
        sr, sc = slice_shape(rows, cols, split, tp)
        offs.append(off)
        off += ((sr + tile - 1) // tile) * ((sc + tile - 1) // tile)
    return offs


def reshard_cast_items(spec, src_tp: int, dst_tp: int, rank: int) -> np.ndarray:
    """Cast items that build rank ``rank``'s packed fp8 shard of the
    ``dst_tp`` split (with packed scale grids) directly from a buffer holding
    the ``src_tp`` bf16 shards rank-major."""
    from . import tc_reshard_cast_items
    views = reshard_views(spec, src_tp, dst_tp, elem_bytes=2, dst_elem_bytes=1)
    return tc_reshard_cast_items(views, scale_offsets(spec, dst_tp), dst_tp, rank)
