"""GPU parity at the launch limits of the block-scaled cast and its inverse.

The full-tile kernels are launched in chunks: the cast at most 2^22 tiles per
launch (with or without the per-tile table), the inverse's quarter-tile
kernel at most 2^20 tiles per launch.  These cases cross those boundaries
with thousands of items that all read one source matrix (a read may be shared;
every item writes its own output), so the output alone takes the memory:
4,195,328 tiles (2^22 + 1024) of codes for the cast, 1,049,600 tiles
(2^20 + 1024) of bf16 for the inverse.  The shared source is compared with
the oracle once, and every item's output must equal the first item's bit for
bit, so a tile taken from the wrong chunk, skipped or written twice shows.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_06007_amd as tc

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
ROWS, TILES_PER_ITEM = 128, 1024
COLS = 128 * TILES_PER_ITEM


def _host(t):
    return t.detach().to("cpu").numpy()


def _shared_source_items(n, dtype, own_scales):
    """n items over one 128 x 131072 source, each writing its own row of 1024
    tiles (codes or bf16).  The cast writes its own 1024 scales per item
    (own_scales); the inverse's items all read the one source's 1024."""
    items = np.zeros(n, dtype=dtype)
    k = np.arange(n, dtype=np.int64)
    items["src_off"] = 0
    items["rows"] = ROWS
    items["cols"] = COLS
    items["src_ld"] = COLS
    items["dst_off"] = k * ROWS * COLS
    items["dst_ld"] = COLS
    items["scale_off"] = k * TILES_PER_ITEM if own_scales else 0
    items["scale_ld"] = TILES_PER_ITEM
    return items


def _items_fit(items, n_src, n_dst, n_scales):
    """Every element an item reads or writes lies inside its buffer (checked
    on the host before any launch)."""
    last = (items["rows"] - 1) * items["src_ld"] + items["cols"]
    assert int((items["src_off"] + last).max()) <= n_src
    last = (items["rows"] - 1) * items["dst_ld"] + items["cols"]
    assert int((items["dst_off"] + last).max()) <= n_dst
    tiles_r = (items["rows"] + 127) // 128
    tiles_c = (items["cols"] + 127) // 128
    assert int((items["scale_off"] + (tiles_r - 1) * items["scale_ld"] + tiles_c).max()) <= n_scales


def _every_item_equals_the_first(out, n, per_item, what):
    first = out[:per_item]
    for k in range(1, n):
        assert torch.equal(out[k * per_item:(k + 1) * per_item], first), (what, k)


@pytest.mark.parametrize("tiled", [True, False])
def test_cast_past_a_launch_of_2_22_tiles(tiled):
    n = (1 << 22) // TILES_PER_ITEM + 1
    items = _shared_source_items(n, tc.CAST_ITEM_DTYPE, own_scales=True)
    print(f"case cast chunks tiled={tiled} items={n} tiles={n * TILES_PER_ITEM}", flush=True)
    src = synth.bf16_normal(ROWS * COLS, 0.02, 4100, device=DEV)
    q = torch.full((n * ROWS * COLS,), 0xEE, dtype=torch.uint8, device=DEV)
    sc = torch.full((n * TILES_PER_ITEM,), -1.0, dtype=torch.float32, device=DEV)
    _items_fit(items, src.numel(), q.numel(), sc.numel())
    wsb = tc.tc_cast_fp8_workspace_tiles(items) if tiled else tc.tc_cast_fp8_workspace(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    plan = tc.tc_cast_fp8_prepare(src, q, items, ws)
    assert plan.tiled == (1 if tiled else 0) and plan.full_tiles == n * TILES_PER_ITEM > (1 << 22)
    tc.tc_cast_fp8_planned(src, q, sc, ws, plan)
    torch.cuda.synchronize()
    want_q, want_s = oracle.cast_fp8_blockscaled(_host(src.view(torch.int16)).view(np.uint16).reshape(ROWS, COLS))
    assert np.array_equal(_host(q[:ROWS * COLS]).reshape(ROWS, COLS), want_q)
    assert np.array_equal(_host(sc[:TILES_PER_ITEM]).view(np.uint32), want_s.reshape(-1).view(np.uint32))
    _every_item_equals_the_first(q, n, ROWS * COLS, "codes")
    _every_item_equals_the_first(sc.view(torch.int32), n, TILES_PER_ITEM, "scales")
    del q, sc, ws, src
    torch.cuda.empty_cache()


def test_inverse_past_a_launch_of_2_20_tiles():
    n = (1 << 20) // TILES_PER_ITEM + 1
    items = _shared_source_items(n, tc.DEQUANT_ITEM_DTYPE, own_scales=False)
    print(f"case inverse chunks items={n} tiles={n * TILES_PER_ITEM}", flush=True)
    # codes and scales the oracle's cast gives for a N(0, 1) source
    bits = _host(synth.bf16_normal(ROWS * COLS, 1.0, 4101, device=DEV).view(torch.int16)).view(np.uint16)
    hq, hs = oracle.cast_fp8_blockscaled(bits.reshape(ROWS, COLS))
    q = torch.from_numpy(np.ascontiguousarray(hq).reshape(-1)).to(DEV)
    sc = torch.from_numpy(np.ascontiguousarray(hs).reshape(-1)).to(DEV)
    y = torch.full((n * ROWS * COLS,), 0x5A5A, dtype=torch.int16, device=DEV).view(torch.bfloat16)
    _items_fit(items, q.numel(), y.numel(), sc.numel())
    ws = torch.empty(tc.tc_dequant_fp8_workspace_tiles(items), dtype=torch.uint8, device=DEV)
    plan = tc.tc_dequant_fp8_prepare(q, y, items, ws)
    assert plan.tiled == 1 and plan.full_tiles == n * TILES_PER_ITEM > (1 << 20)
    tc.tc_dequant_fp8_planned(q, sc, y, ws, plan)
    torch.cuda.synchronize()
    want = oracle.dequant_fp8_blockscaled(hq, hs)
    assert np.array_equal(_host(y[:ROWS * COLS].view(torch.int16)).view(np.uint16).reshape(ROWS, COLS), want)
    _every_item_equals_the_first(y.view(torch.int16), n, ROWS * COLS, "bf16")
    del y, ws, q, sc
    torch.cuda.empty_cache()
