"""Host-side checks of the C-ABI library (CPU only, no kernel launches).

* The library loads and exports every function the public header declares.
* Argument errors are reported before any device work.
* The tensor-parallel builders describe exactly the oracle's numpy slices:
  their fragments, applied by the oracle's byte copier to host buffers,
  reproduce the oracle's shard.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import synth
import paper_2608_06007_amd as tc
from paper_2608_06007_amd import views as tcv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tensorcast_hip.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(tc.lib_path):
        from paper_2608_06007_amd import build
        build.build()
    return tc.load()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tc_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_function(lib):
    names = _declared_functions()
    assert len(names) >= 15
    for name in names:
        assert hasattr(lib, name), name


def test_status_strings(lib):
    assert tc.tc_status_string(0) == "ok"
    assert tc.tc_status_string(5) == "workspace too small"
    assert tc.tc_status_string(6) == "host memory or threads unavailable"


def test_absurd_counts_are_refused_not_wrapped(lib):
    P = ctypes.c_void_p
    huge = 1 << 58                       # sizes for this many would not fit size_t
    assert tc.tc_copy_fragments_workspace(huge) == 0
    assert tc.tc_copy_fragments_workspace_min(huge) == 0
    assert tc.tc_cast_fp8_workspace(huge) == 0
    assert tc.tc_dequant_fp8_workspace(huge) == 0
    assert lib.tc_cast_fp8_blockscaled(P(16), P(16), P(16), P(16), huge, 128, P(4096), 1 << 20, None) == 1
    assert lib.tc_dequant_fp8_blockscaled(P(16), P(16), P(16), P(16), huge, 128, P(4096), 1 << 20, None) == 1
    assert lib.tc_plan_fragments(P(16), huge, P(4096), 1 << 20, None, None) == 1
    assert lib.tc_copy_fragments(P(16), P(16), P(16), huge, P(4096), 1 << 20, None) == 1
    # counts just past the limit (2^33), and task counts past it
    over = (1 << 33) + 1
    assert tc.tc_copy_fragments_workspace(over) == 0 and tc.tc_copy_fragments_workspace(1 << 33) > 0
    assert lib.tc_plan_fragments(P(16), over, P(4096), 1 << 20, None, None) == 1
    assert lib.tc_copy_planned(P(16), P(16), P(4096), 1 << 62, ctypes.c_uint64(over), None) == 1
    assert lib.tc_digest_planned(P(16), 0, P(4096), 1 << 62, ctypes.c_uint64(over), 1, P(16), None) == 1


def test_argument_errors_need_no_gpu(lib):
    P = ctypes.c_void_p
    # gather with a null pool
    assert lib.tc_gather_blocks(None, P(16), 1, P(16), None) == 1
    # zero-length calls are no-ops even with null pointers
    arr = (ctypes.c_uint64 * 1)(4096)
    pool = tc._BlockPool(ctypes.cast(arr, ctypes.POINTER(ctypes.c_uint64)), 1, 4, 64, 64)
    assert lib.tc_gather_blocks(ctypes.byref(pool), None, 0, None, None) == 0
    # stride smaller than the block
    pool_bad = tc._BlockPool(ctypes.cast(arr, ctypes.POINTER(ctypes.c_uint64)), 1, 4, 64, 32)
    assert lib.tc_gather_blocks(ctypes.byref(pool_bad), P(16), 1, P(16), None) == 1
    # too many regions
    big = (ctypes.c_uint64 * 300)(*([4096] * 300))
    pool_big = tc._BlockPool(ctypes.cast(big, ctypes.POINTER(ctypes.c_uint64)), 300, 4, 64, 64)
    assert lib.tc_gather_blocks(ctypes.byref(pool_big), P(16), 1, P(16), None) == 1
    # byte extents beyond 63 bits: a region (blocks x stride), the transfer buffer (n x R x B)
    pool_wide = tc._BlockPool(ctypes.cast(arr, ctypes.POINTER(ctypes.c_uint64)), 1, 1 << 40, 1 << 23, 1 << 23)
    assert lib.tc_gather_blocks(ctypes.byref(pool_wide), P(16), 1, P(16), None) == 1
    pool_huge = tc._BlockPool(ctypes.cast(big, ctypes.POINTER(ctypes.c_uint64)), 64, 4, 1 << 30, 1 << 30)
    assert lib.tc_scatter_blocks(ctypes.byref(pool_huge), P(16), 1 << 27, P(16), None) == 1
    # the staging calls check the pool the same way before any copy (the
    # stager handle is not dereferenced on these paths)
    for bad in (pool_bad, pool_wide):
        assert lib.tc_hydrate_from_host(P(16), ctypes.byref(bad), P(16), 1, P(16), 0, P(16), 1 << 20, None) == 1
        assert lib.tc_publish_to_host(P(16), ctypes.byref(bad), P(16), 1, P(16), 0, P(16), 1 << 20, None) == 1
    nul = (ctypes.c_uint64 * 2)(4096, 0)                 # a null region
    pool_nul = tc._BlockPool(ctypes.cast(nul, ctypes.POINTER(ctypes.c_uint64)), 2, 4, 64, 64)
    assert lib.tc_hydrate_from_host(P(16), ctypes.byref(pool_nul), P(16), 1, P(16), 0, P(16), 1 << 20, None) == 1
    assert lib.tc_gather_blocks(ctypes.byref(pool_nul), P(16), 1, P(16), None) == 1
    # fragments: workspace too small, negative count
    assert lib.tc_copy_fragments(P(16), P(16), P(16), 10, P(4096), 8, None) == 5
    assert lib.tc_copy_fragments(P(16), P(16), P(16), 10, P(4100), 1 << 20, None) == 1  # misaligned
    assert lib.tc_copy_fragments(P(16), P(16), P(16), -1, P(16), 1 << 20, None) == 1
    assert lib.tc_copy_fragments(None, None, None, 0, None, 0, None) == 0
    # a task count the workspace's table cannot hold is refused before any launch
    assert lib.tc_copy_planned(P(16), P(16), P(4096), 256 + 32 * 10, ctypes.c_uint64(11), None) == 5
    assert lib.tc_copy_planned(P(16), P(16), P(4096), 100, ctypes.c_uint64(1), None) == 5
    # cast: tile other than 128
    assert lib.tc_cast_fp8_blockscaled(P(16), P(16), P(16), P(16), 1, 64, P(16), 1 << 20, None) == 1
    assert lib.tc_cast_fp8_scaled(P(16), -5, ctypes.c_float(1.0), P(16), None) == 1
    assert tc.tc_copy_fragments_workspace(1000) >= 24 * 1001
    # digests: negative count, unknown side, misaligned digest array, no
    # destination with work to do, task count beyond the workspace
    U64 = ctypes.c_uint64
    assert lib.tc_copy_planned_digest(P(16), P(16), P(4096), 1 << 20, U64(1), -1, P(16), None) == 1
    assert lib.tc_digest_planned(P(16), 2, P(4096), 1 << 20, U64(1), 1, P(16), None) == 1
    assert lib.tc_digest_planned(P(16), 0, P(4096), 1 << 20, U64(1), 1, P(12), None) == 1
    assert lib.tc_copy_planned_digest(P(16), None, P(4096), 1 << 20, U64(1), 1, P(16), None) == 1
    assert lib.tc_copy_planned_digest(P(16), P(16), P(4096), 4096, U64(1000), 1, P(16), None) == 5
    assert lib.tc_copy_planned_digest(None, None, None, 0, U64(0), 0, None, None) == 0
    # staging: bad ring shapes and flags are refused before any HIP call
    h = ctypes.c_void_p(0)
    assert lib.tc_stager_create(0, 1, 0, ctypes.byref(h)) == 1        # one slot cannot overlap
    assert lib.tc_stager_create(100, 2, 0, ctypes.byref(h)) == 1      # slot below 4 KiB
    assert lib.tc_stager_create(0, -1, 0, ctypes.byref(h)) == 1
    assert lib.tc_stager_create(0, 0, 0, None) == 1
    assert lib.tc_stager_destroy(None) == 0
    assert lib.tc_stage_h2d(None, P(16), P(16), 10, 0, None) == 1
    assert lib.tc_stage_d2h(None, P(16), P(16), 10, 0, None) == 1
    # cast items are checked on the host before anything is staged
    items = np.zeros(1, dtype=tc.CAST_ITEM_DTYPE)
    items[0] = (0, 128, 256, 100, 0, 256, 0, 2)          # src_ld < cols
    assert lib.tc_cast_fp8_blockscaled(P(16), P(16), P(16), items.ctypes.data, 1, 128, P(4096),
                                       1 << 20, None) == 1
    items[0] = (0, 128, 256, 256, 0, 256, 0, 1)          # scale_ld < tile columns
    assert lib.tc_cast_fp8_blockscaled(P(16), P(16), P(16), items.ctypes.data, 1, 128, P(4096),
                                       1 << 20, None) == 1
    assert tc.tc_cast_fp8_workspace(10) >= 8 * 11
    # inverse cast: tile and geometry checks before anything is staged
    ditems = np.zeros(1, dtype=tc.DEQUANT_ITEM_DTYPE)
    ditems[0] = (0, 128, 256, 256, 0, 256, 0, 2)
    assert lib.tc_dequant_fp8_blockscaled(P(16), P(16), P(16), ditems.ctypes.data, 1, 64, P(4096),
                                          1 << 20, None) == 1
    ditems[0] = (0, 128, 256, 200, 0, 256, 0, 2)          # code row stride < cols
    assert lib.tc_dequant_fp8_blockscaled(P(16), P(16), P(16), ditems.ctypes.data, 1, 128, P(4096),
                                          1 << 20, None) == 1
    assert lib.tc_dequant_fp8_blockscaled(P(16), P(16), P(16), ditems.ctypes.data, 1, 128, P(4096),
                                          16, None) == 5


def test_new_entry_points_check_arguments_without_a_gpu(lib):
    """The asynchronous planning, prepared casts and IPC calls refuse bad
    arguments on the host, before anything is enqueued."""
    P = ctypes.c_void_p
    U64 = ctypes.c_uint64
    # planning without waiting: the same argument checks as tc_plan_fragments
    assert lib.tc_plan_fragments_async(P(16), -1, P(4096), 1 << 20, None) == 1
    assert lib.tc_plan_fragments_async(P(16), 10, P(4100), 1 << 20, None) == 1   # misaligned
    assert lib.tc_plan_fragments_async(P(16), 10, P(4096), 8, None) == 5        # too small
    assert lib.tc_plan_fragments_async(None, 0, None, 0, None) == 0
    assert lib.tc_plan_status(None, 1 << 20, None, None) == 1
    assert lib.tc_plan_status(P(4100), 1 << 20, None, None) == 1
    # a copy that takes its count from the plan still needs a task table
    assert lib.tc_copy_planned(P(16), P(16), P(4096), 100, U64((1 << 64) - 1), None) == 5
    assert lib.tc_copy_planned(None, P(16), P(4096), 1 << 20, U64((1 << 64) - 1), None) == 1
    # prepared casts
    plan = tc.TilePlan()
    item = np.zeros(1, dtype=tc.CAST_ITEM_DTYPE)
    item[0] = (0, 128, 128, 128, 0, 128, 0, 1)
    it = item.ctypes.data
    assert lib.tc_cast_fp8_prepare(P(16), P(16), it, 1, 128, P(4096), 1 << 20, None, None) == 1
    assert lib.tc_cast_fp8_prepare(P(16), P(16), it, 1, 64, P(4096), 1 << 20, ctypes.byref(plan), None) == 1
    assert lib.tc_cast_fp8_prepare(P(16), P(16), it, 1, 128, P(4096), 64, ctypes.byref(plan), None) == 5
    assert lib.tc_cast_fp8_prepare(P(17), P(16), it, 1, 128, P(4096), 1 << 20, ctypes.byref(plan), None) == 1
    bad = item.copy()
    bad[0]["src_ld"] = 100                                   # row stride below the width
    assert lib.tc_cast_fp8_prepare(P(16), P(16), bad.ctypes.data, 1, 128, P(4096), 1 << 20,
                                   ctypes.byref(plan), None) == 1
    assert lib.tc_dequant_fp8_prepare(P(16), P(17), it, 1, 128, P(4096), 1 << 20, ctypes.byref(plan), None) == 1
    # a plan made for 16-byte-aligned bases refuses bases of another alignment
    plan = tc.TilePlan(1, 1, 0, 0, 0)
    assert lib.tc_cast_fp8_planned(P(34), P(64), P(128), P(4096), 1 << 20, ctypes.byref(plan), None) == 1
    assert lib.tc_cast_fp8_planned(P(32), P(64), P(130), P(4096), 1 << 20, ctypes.byref(plan), None) == 1
    assert lib.tc_cast_fp8_planned(P(32), P(64), P(128), P(4096), 64, ctypes.byref(plan), None) == 5
    assert lib.tc_cast_fp8_planned(P(32), P(64), P(128), P(4096), 1 << 20, None, None) == 1
    empty = tc.TilePlan(0, 0, 0, 0, 0)
    assert lib.tc_cast_fp8_planned(None, None, None, None, 0, ctypes.byref(empty), None) == 0
    assert lib.tc_dequant_fp8_planned(P(34), P(128), P(64), P(4096), 1 << 20, ctypes.byref(plan), None) == 1
    # a plan that reads a per-tile table needs room for it; the flag is 0 or 1
    base = tc.tc_cast_fp8_workspace(1)
    tiled = tc.TilePlan(1, 10, 0, 0, 0, 1, 0)
    assert lib.tc_cast_fp8_planned(P(32), P(64), P(128), P(4096), base + 32 * 9, ctypes.byref(tiled), None) == 5
    assert lib.tc_dequant_fp8_planned(P(32), P(128), P(64), P(4096), base + 32 * 9, ctypes.byref(tiled),
                                      None) == 5
    tiled.full_tiles = (1 << 63) + 1                          # no wrap in the size check
    assert lib.tc_cast_fp8_planned(P(32), P(64), P(128), P(4096), 1 << 30, ctypes.byref(tiled), None) == 5
    odd = tc.TilePlan(1, 1, 0, 0, 0, 2, 0)
    assert lib.tc_cast_fp8_planned(P(32), P(64), P(128), P(4096), 1 << 20, ctypes.byref(odd), None) == 1
    assert lib.tc_dequant_fp8_planned(P(32), P(128), P(64), P(4096), 1 << 20, ctypes.byref(odd), None) == 1
    # IPC: null arguments, and handles that describe impossible ranges
    h = tc._IpcHandle()
    out = ctypes.c_void_p(0)
    assert lib.tc_ipc_export(None, 16, ctypes.byref(h)) == 1
    assert lib.tc_ipc_export(P(4096), 16, None) == 1
    assert lib.tc_ipc_open(None, ctypes.byref(out)) == 1
    h.alloc_bytes = 1 << 31                                  # allocations of 2 GiB or more are refused
    assert lib.tc_ipc_open(ctypes.byref(h), ctypes.byref(out)) == 1
    h.alloc_bytes, h.offset, h.bytes = 4096, 4000, 200       # a range past its allocation
    assert lib.tc_ipc_open(ctypes.byref(h), ctypes.byref(out)) == 1
    assert lib.tc_ipc_close(None, P(4096)) == 1
    assert tc.IPC_HANDLE_BYTES == 88


def test_tile_table_workspace_sizes(lib):
    """The workspace that also holds the per-tile table: the items' own
    workspace plus 32 bytes for each full 128 x 128 tile, rounded up to 256
    bytes; 0 for items it cannot size."""
    items = np.zeros(3, dtype=tc.CAST_ITEM_DTYPE)
    items[0] = (0, 300, 520, 520, 0, 520, 0, 5)         # 2 x 4 full tiles
    items[1] = (0, 127, 4096, 4096, 0, 4096, 0, 32)     # no full row of tiles
    items[2] = (0, 1024, 1024, 1024, 0, 1024, 0, 8)     # 8 x 8
    for fn, dt, base in ((tc.tc_cast_fp8_workspace_tiles, tc.CAST_ITEM_DTYPE, tc.tc_cast_fp8_workspace),
                         (tc.tc_dequant_fp8_workspace_tiles, tc.DEQUANT_ITEM_DTYPE,
                          tc.tc_dequant_fp8_workspace)):
        it = items.astype(dt)
        assert fn(it) == base(3) + (72 * 32 + 255) // 256 * 256
        assert fn(it[1:2]) == base(1)
        assert fn(it[:0]) == base(0)
        bad = it.copy()
        bad[1]["rows"] = -1
        assert fn(bad) == 0
    P = ctypes.c_void_p
    assert lib.tc_cast_fp8_workspace_tiles(None, 2) == 0
    assert lib.tc_dequant_fp8_workspace_tiles(P(items.ctypes.data), -1) == 0


def test_binding_refuses_wrong_dtypes_before_any_call(lib):
    """Dtype checks in the binding run before a device address is taken, so
    they need no GPU: ids must be int32 (the library reads 4-byte ids),
    fragment rows 64-bit integers, and the scaled cast's source 2-byte
    elements with a byte of output each."""
    import torch
    regions = [4096, 8192]                                # raw addresses: never dereferenced
    with pytest.raises(ValueError, match="int32"):
        tc.tc_gather_blocks(regions, 4, 64, 64, torch.zeros(2, dtype=torch.int64), 12288)
    with pytest.raises(ValueError, match="int32"):
        tc.tc_scatter_blocks(regions, 4, 64, 64, torch.zeros(2, dtype=torch.int16), 12288)
    with pytest.raises(ValueError, match="int32"):
        tc.tc_hydrate_from_host(16, regions, 4, 64, 64, torch.zeros(2, dtype=torch.float32),
                                np.zeros(256, np.uint8), 4096)
    with pytest.raises(ValueError, match="uint64/int64"):
        tc.tc_copy_fragments(4096, 8192, torch.zeros((2, 3), dtype=torch.float64), 16384)
    with pytest.raises(ValueError, match="uint64/int64"):
        tc.tc_plan_fragments(torch.zeros(48, dtype=torch.uint8), 16384)
    with pytest.raises(ValueError, match="2-byte"):
        tc.tc_cast_fp8_scaled(torch.zeros(8, dtype=torch.uint8), 1.0, torch.zeros(8, dtype=torch.uint8))
    with pytest.raises(ValueError, match="dst too small"):
        tc.tc_cast_fp8_scaled(torch.zeros(8, dtype=torch.bfloat16), 1.0, torch.zeros(4, dtype=torch.uint8))


def test_validate_flag_roundtrip(lib):
    tc.tc_set_validate(True)
    assert tc.tc_get_validate()
    tc.tc_set_validate(False)
    assert not tc.tc_get_validate()


SPEC = synth.spec_scaled(layers=2, hidden=256, q_heads=4, kv_heads=2, head_dim=64, mlp=384)


@pytest.mark.parametrize("tp", [1, 2, 4, 8])
def test_tp_fragments_reproduce_oracle_shard(lib, tp):
    n = synth.spec_elems(SPEC)
    rng = np.random.default_rng(20)
    stream = rng.integers(0, 1 << 16, size=n, dtype=np.uint64).astype(np.uint16)
    src = stream.view(np.uint8)
    v = tcv.stream_views(SPEC, tp)
    for rank in range(tp):
        frags = tc.tc_tp_fragments(v, tp, rank)
        dst = np.full(tcv.shard_elems(SPEC, tp) * 2, 0xEE, dtype=np.uint8)
        oracle.copy_fragments(src, dst, frags)
        want = oracle.tp_shard(stream, SPEC, tp, rank)
        assert np.array_equal(dst.view(np.uint16), want)
        d = frags[:, 1].astype(np.int64)                 # ascending, no holes
        assert d[0] == 0 and np.array_equal(d[1:], d[:-1] + frags[:-1, 2].astype(np.int64))


def test_tp_fragments_merge_contiguous_rows(lib):
    # row-split slices are contiguous runs: one fragment per matrix;
    # column-split slices need one fragment per row
    v = tcv.stream_views(SPEC, 8)
    frags = tc.tc_tp_fragments(v, 8, 3)
    per_layer = 5 + 256 + 256          # q k v gate up + o rows + down rows
    assert len(frags) == 2 * per_layer
    assert tc.tc_tp_fragment_count(v, 8, 3) == len(frags)


def test_tp_builder_rejects_bad_views(lib):
    v = tcv.stream_views(SPEC, 8)
    with pytest.raises(tc.TcError):
        tc.tc_tp_fragments(v, 3, 0)          # 256 rows not divisible by 3
    with pytest.raises(tc.TcError):
        tc.tc_tp_fragments(v, 8, 8)          # rank out of range
    bad = v.copy()
    bad[0]["src_ld"] = 10                    # ld < cols
    with pytest.raises(tc.TcError):
        tc.tc_tp_fragments(bad, 8, 0)


def test_cast_items_describe_the_slices(lib):
    tp, rank = 4, 1
    items = tcv.cast_items(SPEC, tp, rank)
    n = synth.spec_elems(SPEC)
    stream = np.arange(n, dtype=np.int64)
    off = 0
    q_off = 0
    s_off = 0
    for it, (_, rows, cols, split) in zip(items, SPEC):
        w = stream[off:off + rows * cols].reshape(rows, cols)
        off += rows * cols
        sl = oracle.tp_slice(w, split, tp, rank)
        assert (it["rows"], it["cols"]) == sl.shape
        # element [0][0] and the row stride of the slice inside the stream
        assert it["src_off"] == sl[0, 0]
        if sl.shape[0] > 1:
            assert it["src_ld"] == sl[1, 0] - sl[0, 0]
        assert it["dst_off"] == q_off and it["dst_ld"] == sl.shape[1]
        assert it["scale_off"] == s_off and it["scale_ld"] == (sl.shape[1] + 127) // 128
        q_off += sl.size
        s_off += ((sl.shape[0] + 127) // 128) * ((sl.shape[1] + 127) // 128)


@pytest.mark.parametrize("src_tp,dst_tp", [(8, 4), (4, 8), (8, 1), (1, 8), (2, 8), (8, 8), (4, 2)])
def test_reshard_fragments_reproduce_oracle_shard(lib, src_tp, dst_tp):
    """Source = the src_tp oracle shards back to back; the builder's fragments,
    applied with the oracle's byte copier, must give the oracle's dst shard."""
    n = synth.spec_elems(SPEC)
    rng = np.random.default_rng(21)
    stream = rng.integers(0, 1 << 16, size=n, dtype=np.uint64).astype(np.uint16)
    src = np.concatenate([oracle.tp_shard(stream, SPEC, src_tp, r) for r in range(src_tp)])
    views = tcv.reshard_views(SPEC, src_tp, dst_tp)
    for rank in range(dst_tp):
        frags = tc.tc_reshard_fragments(views, dst_tp, rank)
        dst = np.full(tcv.shard_elems(SPEC, dst_tp), 0xBEEF, dtype=np.uint16)
        oracle.copy_fragments(src.view(np.uint8), dst.view(np.uint8), frags)
        assert np.array_equal(dst, oracle.tp_shard(stream, SPEC, dst_tp, rank))
        # the list ascends in destination and tiles the shard without holes,
        # so a plan keeps its order
        d = frags[:, 1].astype(np.int64)
        ln = frags[:, 2].astype(np.int64)
        assert d[0] == 0 and np.array_equal(d[1:], d[:-1] + ln[:-1])
        assert int(ln.sum()) == 2 * tcv.shard_elems(SPEC, dst_tp)


def test_reshard_round_trip_and_fragment_counts(lib):
    """TP8 -> TP4 -> TP8 gives back every TP8 shard; a row split needs one
    fragment per overlapping source rank, a column split one per row."""
    n = synth.spec_elems(SPEC)
    stream = np.arange(n, dtype=np.uint64).astype(np.uint16) ^ np.uint16(0x5A5A)
    tp8 = np.concatenate([oracle.tp_shard(stream, SPEC, 8, r) for r in range(8)])
    tp4 = []
    for r in range(4):
        dst = np.zeros(tcv.shard_elems(SPEC, 4), dtype=np.uint16)
        oracle.copy_fragments(tp8.view(np.uint8), dst.view(np.uint8),
                              tc.tc_reshard_fragments(tcv.reshard_views(SPEC, 8, 4), 4, r))
        tp4.append(dst)
    tp4 = np.concatenate(tp4)
    for r in range(8):
        dst = np.zeros(tcv.shard_elems(SPEC, 8), dtype=np.uint16)
        oracle.copy_fragments(tp4.view(np.uint8), dst.view(np.uint8),
                              tc.tc_reshard_fragments(tcv.reshard_views(SPEC, 4, 8), 8, r))
        assert np.array_equal(dst, tp8.reshape(8, -1)[r])
    # per layer: q k v gate up -> 2 source ranks each; o, down -> 2 x 256 rows
    assert tc.tc_reshard_fragment_count(tcv.reshard_views(SPEC, 8, 4), 4, 1) == 2 * (5 * 2 + 2 * 256 * 2)
    with pytest.raises(tc.TcError):
        tc.tc_reshard_fragments(tcv.reshard_views(SPEC, 8, 3), 3, 0)   # 3 does not divide


def test_header_compiles_as_plain_c(tmp_path):
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "abi.c"
    src.write_text('#include "tensorcast_hip.h"\nint main(void) { return TC_OK; }\n')
    r = subprocess.run([gcc, "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-D__HIP_PLATFORM_AMD__",
                        f"-I{os.path.dirname(HEADER)}", "-I/opt/rocm/include", str(src)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_c_program_links_against_the_library(tmp_path):
    """tests/c_abi/abi_demo.c builds with a plain C compiler and every library
    symbol it calls resolves at link time (running it needs a GPU)."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    libdir = os.path.join(root, "paper_2608_06007_amd")
    exe = tmp_path / "abi_demo"
    r = subprocess.run([gcc, "-std=c99", "-O1", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
                        f"-I{os.path.dirname(HEADER)}", "-I/opt/rocm/include",
                        os.path.join(root, "tests", "c_abi", "abi_demo.c"), "-o", str(exe),
                        f"-L{libdir}", "-ltchip", "-L/opt/rocm/lib", "-lamdhip64",
                        "-Wl,--no-undefined", "-Wl,--no-allow-shlib-undefined"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    assert exe.exists()


# Dimensions that are multiples of 128 x tp for tp up to 8, small enough for the oracle.
SPEC_TILED = synth.spec_scaled(layers=1, hidden=1024, q_heads=8, kv_heads=8, head_dim=128, mlp=2048)


def _apply_cast_items_with_oracle(src_bits, items, q_size, s_size):
    """Cast every item's sub-matrix with the oracle and place codes and scales
    where the item says (a CPU stand-in for the cast kernel's addressing)."""
    q = np.full(q_size, 0xEE, np.uint8)
    sc = np.full(s_size, np.nan, np.float32)
    for it in items:
        rows, cols = int(it["rows"]), int(it["cols"])
        so, sld = int(it["src_off"]), int(it["src_ld"])
        m = np.lib.stride_tricks.as_strided(src_bits[so:], shape=(rows, cols), strides=(2 * sld, 2))
        codes, scales = oracle.cast_fp8_blockscaled(np.ascontiguousarray(m))
        do, dld = int(it["dst_off"]), int(it["dst_ld"])
        for r in range(rows):
            q[do + r * dld:do + r * dld + cols] = codes[r]
        s0, sl = int(it["scale_off"]), int(it["scale_ld"])
        for r in range(scales.shape[0]):
            sc[s0 + r * sl:s0 + r * sl + scales.shape[1]] = scales[r]
    return q, sc


@pytest.mark.parametrize("src_tp,dst_tp,rank", [(8, 4, 1), (4, 8, 6), (8, 1, 0), (1, 8, 3), (2, 4, 2),
                                                 (8, 8, 5)])
def test_reshard_cast_items_reproduce_the_oracle_cast(lib, src_tp, dst_tp, rank):
    """Items built for a reshard into fp8, applied by the oracle, equal the
    oracle's cast of the destination rank's slices of the full weights."""
    spec = SPEC_TILED
    n = synth.spec_elems(spec)
    rng = np.random.default_rng(21)
    stream = (rng.standard_normal(n).astype(np.float32) * 0.02).view(np.uint32) >> 16
    stream = stream.astype(np.uint16)
    # source buffer: the src_tp shards, rank-major
    src = np.concatenate([oracle.tp_shard(stream, spec, src_tp, r) for r in range(src_tp)])
    items = tcv.reshard_cast_items(spec, src_tp, dst_tp, rank)
    q_size = tcv.shard_elems(spec, dst_tp)
    s_size = tcv.scale_elems(spec, dst_tp)
    q, sc = _apply_cast_items_with_oracle(src, items, q_size, s_size)
    # the oracle's cast of each destination slice, packed the same way
    want_q, want_s = [], []
    off = 0
    for (_n, rows, cols, split) in spec:
        w = stream[off:off + rows * cols].reshape(rows, cols)
        off += rows * cols
        codes, scales = oracle.cast_fp8_blockscaled(
            np.ascontiguousarray(oracle.tp_slice(w, split, dst_tp, rank)))
        want_q.append(codes.reshape(-1))
        want_s.append(scales.reshape(-1))
    assert np.array_equal(q, np.concatenate(want_q))
    assert np.array_equal(sc.view(np.uint32), np.concatenate(want_s).view(np.uint32))


def test_reshard_cast_items_refuse_tiles_across_sources(lib):
    # 192 rows from 3 source ranks of 64 rows: a destination tile would span two sources
    bad = [((0, 192 * 256 * 2 // 3, 2 * 192 * 256 * 2 // 3), 192, 256, 2, tc.SPLIT_ROWS, 0)]
    with pytest.raises(tc.TcError):
        tc.tc_reshard_cast_item_count(bad, 1, 0)
    # odd source offsets cannot hold bf16
    odd = [((1,), 128, 128, 2, tc.SPLIT_NONE, 0)]
    with pytest.raises(tc.TcError):
        tc.tc_reshard_cast_item_count(odd, 1, 0)
    # fp32 views are not castable
    f32 = [((0,), 128, 128, 4, tc.SPLIT_NONE, 0)]
    with pytest.raises(tc.TcError):
        tc.tc_reshard_cast_item_count(f32, 1, 0)


def test_missing_library_fails_loudly():
    """Without the HIP library every entry point raises: there is no CPU
    fallback.  Run in a fresh interpreter with the library path pointed at a
    file that does not exist."""
    import subprocess
    import sys
    code = ("import paper_2608_06007_amd as tc\n"
            "tc.lib_path = '/nonexistent/libtchip.so'\n"
            "try:\n"
            "    tc.tc_copy_fragments_workspace(10)\n"
            "except RuntimeError as e:\n"
            "    print('raised:', e)\n"
            "else:\n"
            "    print('no error')\n")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.startswith("raised:") and "missing" in r.stdout
