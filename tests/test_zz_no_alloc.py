"""GPU: the no-allocation block-scaled cast against the workspace one.

tc_cast_fp8_blockscaled_noalloc keeps its tile table in the library's fixed
device array instead of a caller workspace.  Two calls in a row through the
C ABI -- the second with a smaller item list and matrix, so stale table
entries of the first call would show -- must give the same codes and scales,
bit for bit, as tc_cast_fp8_blockscaled on the same inputs; an item count
above the array's limit is refused before anything is enqueued.
"""
import ctypes

import numpy as np
import pytest
import torch

import synth
import paper_2608_06007_amd as tc

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
MAX_ITEMS = 4096


def _lib():
    L = tc.load()
    P = ctypes.c_void_p
    L.tc_cast_fp8_blockscaled_noalloc.argtypes = [P, P, P, P, ctypes.c_int64, ctypes.c_int32, P]
    L.tc_cast_fp8_blockscaled_noalloc.restype = ctypes.c_int
    return L


def _items(n_items, rows, cols, ld):
    """n_items row bands of a rows x cols matrix (row stride ld elements),
    each cast into its own dense code block and scale grid."""
    band = rows // n_items
    tcn = (cols + 127) // 128
    items = np.zeros(n_items, dtype=tc.CAST_ITEM_DTYPE)
    q_off = s_off = 0
    for i in range(n_items):
        r = band if i < n_items - 1 else rows - band * (n_items - 1)
        items[i] = (i * band * ld, r, cols, ld, q_off, cols, s_off, tcn)
        q_off += r * cols
        s_off += ((r + 127) // 128) * tcn
    return items, q_off, s_off


def _run_both(L, items, n_codes, n_scales, x, stream):
    q_ref = torch.full((n_codes,), 0xEE, dtype=torch.uint8, device=DEV)
    s_ref = torch.full((n_scales,), -1.0, dtype=torch.float32, device=DEV)
    ws = torch.empty(tc.tc_cast_fp8_workspace(len(items)), dtype=torch.uint8, device=DEV)
    tc.tc_cast_fp8_blockscaled(x, q_ref, s_ref, items, ws, stream=stream)
    q = torch.full_like(q_ref, 0xEE)
    s = torch.full_like(s_ref, -1.0)
    st = L.tc_cast_fp8_blockscaled_noalloc(x.data_ptr(), q.data_ptr(), s.data_ptr(), items.ctypes.data,
                                           len(items), 128, stream.cuda_stream)
    assert st == 0, tc.tc_status_string(st)
    stream.synchronize()
    assert torch.equal(q, q_ref)
    assert torch.equal(s.view(torch.int32), s_ref.view(torch.int32))


def test_noalloc_cast_matches_workspace_cast_twice_then_smaller():
    L = _lib()
    stream = torch.cuda.Stream()
    # first call: 300 items (8 table chunks) of 136 rows over a 40800 x 1000
    # matrix with a padded row stride: full tiles, and partial tiles at every
    # band's bottom and at the right edge
    rows, cols, ld = 40800, 1000, 1040
    x = synth.bf16_normal(rows * ld, 0.02, 4242, device=DEV)
    items, nq, ns = _items(300, rows, cols, ld)
    print("case: noalloc cast, 300 items, 40800 x 1000", flush=True)
    _run_both(L, items, nq, ns, x, stream)
    # second call, smaller: 5 items over 640 x 384 (whole tiles only)
    rows2, cols2 = 640, 384
    x2 = synth.bf16_normal(rows2 * cols2, 1.0, 4243, device=DEV)
    items2, nq2, ns2 = _items(5, rows2, cols2, cols2)
    print("case: noalloc cast, 5 items, 640 x 384", flush=True)
    _run_both(L, items2, nq2, ns2, x2, stream)


def test_noalloc_cast_refuses_too_many_items():
    L = _lib()
    items = np.zeros(MAX_ITEMS + 1, dtype=tc.CAST_ITEM_DTYPE)
    st = L.tc_cast_fp8_blockscaled_noalloc(16, 16, 16, items.ctypes.data, len(items), 128, None)
    assert st == 5  # TC_ERR_WORKSPACE, nothing enqueued
    assert L.tc_cast_fp8_blockscaled_noalloc(16, 16, 16, items.ctypes.data, 1, 64, None) == 1
