"""GPU parity: bf16 -> fp8 E4M3 casts.

HIP path through the C ABI against the CPU oracle, bit for bit (codes and
scale bits): every bf16 pattern at many scales, block-scaled matrices with
ragged and strided tiles and special tiles, a TP=8 shard of 70B-shaped
weights on a few layers in full and at full size on sampled tiles.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_06007_amd as tc
from paper_2608_06007_amd import views as tcv

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
ALL_BF16 = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)


def _host(t):
    return t.detach().to("cpu").numpy()


def _to_dev_bits(bits: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.bfloat16)


def _gpu_scaled(bits: np.ndarray, scale: float) -> np.ndarray:
    x = _to_dev_bits(bits)
    q = torch.empty(x.numel(), dtype=torch.uint8, device=DEV)
    tc.tc_cast_fp8_scaled(x, scale, q)
    torch.cuda.synchronize()
    return _host(q)


def test_every_bf16_pattern_scale_one():
    got = _gpu_scaled(ALL_BF16, 1.0)
    want = oracle.cast_fp8_scaled(ALL_BF16, 1.0)
    assert np.array_equal(got, want)


def test_every_bf16_pattern_many_scales():
    rng = np.random.default_rng(50)
    bits = np.concatenate([rng.integers(0x00800000, 0x7F000000, size=48, dtype=np.int64),
                           rng.integers(1, 0x00800000, size=8, dtype=np.int64),
                           (np.arange(-12, 13) + 127) << 23]).astype(np.uint32)
    for s in bits.view(np.float32):
        got = _gpu_scaled(ALL_BF16, float(s))
        want = oracle.cast_fp8_scaled(ALL_BF16, float(s))
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, (float(s), [(hex(int(ALL_BF16[i])), hex(got[i]), hex(want[i])) for i in bad[:5]])


def test_scaled_odd_sizes_and_offsets():
    rng = np.random.default_rng(51)
    bits = rng.integers(0, 1 << 16, size=10007, dtype=np.int64).astype(np.uint16)
    x = _to_dev_bits(bits)
    for start, stop in [(0, 10007), (1, 10000), (3, 4), (5, 5)]:
        xs = x[start:stop]
        q = torch.empty(xs.numel() + 3, dtype=torch.uint8, device=DEV)[1:1 + xs.numel()]
        tc.tc_cast_fp8_scaled(xs, 0.37, q)
        torch.cuda.synchronize()
        assert np.array_equal(_host(q), oracle.cast_fp8_scaled(bits[start:stop], 0.37))


# ---------------------------------------------------------------------------

def _bits_from_float(a: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _cast_matrices(src_bits_1d: np.ndarray, mats, code_pad=0, scale_pad=0):
    """mats: list of (src_off, rows, cols, src_ld) in bf16 elements of the
    1-D source.  Codes packed row-major (row stride cols + code_pad), scale
    grids packed (row stride tiles_c + scale_pad).  Returns GPU and oracle
    results per matrix."""
    items = np.zeros(len(mats), dtype=tc.CAST_ITEM_DTYPE)
    q_off = s_off = 0
    for k, (so, rows, cols, ld) in enumerate(mats):
        tr, tcn = (rows + 127) // 128, (cols + 127) // 128
        items[k] = (so, rows, cols, ld, q_off, cols + code_pad, s_off, tcn + scale_pad)
        q_off += rows * (cols + code_pad)
        s_off += tr * (tcn + scale_pad)
    src = _to_dev_bits(src_bits_1d)
    # the item table alone (tiles found by searching the items), then with
    # the per-tile table as well: both against the oracle
    for ws_bytes in (tc.tc_cast_fp8_workspace(len(mats)), tc.tc_cast_fp8_workspace_tiles(items)):
        hq, hs = _cast_and_check(src, src_bits_1d, items, mats, q_off, s_off, ws_bytes)
    return hq, hs


def _cast_and_check(src, src_bits_1d, items, mats, q_off, s_off, ws_bytes):
    dst = torch.full((max(q_off, 1),), 0xCC, dtype=torch.uint8, device=DEV)
    scales = torch.full((max(s_off, 1),), -7.0, dtype=torch.float32, device=DEV)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
    tc.tc_cast_fp8_blockscaled(src, dst, scales, items, ws)
    torch.cuda.synchronize()
    hq, hs = _host(dst), _host(scales)
    for k, (so, rows, cols, ld) in enumerate(mats):
        it = items[k]
        view = np.lib.stride_tricks.as_strided(src_bits_1d[so:], shape=(rows, cols), strides=(2 * ld, 2))
        q, s = oracle.cast_fp8_blockscaled(view)
        gq = np.lib.stride_tricks.as_strided(hq[it["dst_off"]:], shape=(rows, cols),
                                             strides=(int(it["dst_ld"]), 1))
        tr, tcn = s.shape
        gs = np.lib.stride_tricks.as_strided(hs[it["scale_off"]:], shape=(tr, tcn),
                                             strides=(4 * int(it["scale_ld"]), 4))
        assert np.array_equal(gs.view(np.uint32), s.view(np.uint32)), f"scales of matrix {k}"
        if not np.array_equal(gq, q):
            bad = np.argwhere(gq != q)
            r, c = bad[0]
            raise AssertionError(f"matrix {k}: {len(bad)} codes differ, first at {(r, c)}: "
                                 f"x={hex(int(view[r, c]))} gpu={hex(int(gq[r, c]))} oracle={hex(int(q[r, c]))}")
    return hq, hs


def test_blockscaled_ragged_strided_and_offsets():
    rng = np.random.default_rng(52)
    a = rng.normal(0, 0.02, size=600 * 700).astype(np.float32)
    bits = _bits_from_float(a)
    mats = [(0, 256, 384, 384),            # whole tiles, packed
            (0, 300, 200, 700),            # ragged rows and cols, strided rows
            (8, 128, 128, 700),            # aligned strided tile
            (3, 130, 129, 700),            # unaligned source (odd element offset)
            (1000, 1, 1, 1),               # single element
            (2000, 5, 300, 301)]           # odd row stride
    _cast_matrices(bits, mats)
    _cast_matrices(bits, mats, code_pad=5, scale_pad=2)     # unaligned code rows


def test_workspace_short_of_the_tile_table_takes_the_search():
    """A workspace with room for the item table but not for every full
    tile's entry: prepare falls back to the item search (plan.tiled == 0)
    for the cast and its inverse, and both still match the oracle; one
    more byte and the table is used."""
    rng = np.random.default_rng(56)
    bits = _bits_from_float(rng.normal(0, 0.02, size=520 * 400).astype(np.float32))
    # 2 x 3 and 1 x 2 full tiles, every row vector-aligned (bf16 pitch a multiple
    # of 16 B, code pitch of 8 B), so all eight go through the table
    mats = [(0, 256, 384, 400), (256 * 400, 130, 264, 264)]
    items = np.zeros(len(mats), dtype=tc.CAST_ITEM_DTYPE)
    q_off = s_off = 0
    for k, (so, rows, cols, ld) in enumerate(mats):
        tr, tcn = (rows + 127) // 128, (cols + 127) // 128
        items[k] = (so, rows, cols, ld, q_off, cols, s_off, tcn)
        q_off += rows * cols
        s_off += tr * tcn
    base, full = tc.tc_cast_fp8_workspace(len(mats)), tc.tc_cast_fp8_workspace_tiles(items)
    assert full == base + 256                                  # 8 entries of 32 B, rounded up
    src = _to_dev_bits(bits)
    q = torch.empty(q_off, dtype=torch.uint8, device=DEV)
    ditems = items.astype(tc.DEQUANT_ITEM_DTYPE)
    ditems["src_off"], ditems["src_ld"] = items["dst_off"], items["dst_ld"]
    ditems["dst_ld"] = items["dst_ld"]
    y = torch.empty(q_off, dtype=torch.bfloat16, device=DEV)
    for ws_bytes, want_tiled in ((full - 1, 0), (full, 1)):
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
        plan = tc.tc_cast_fp8_prepare(src, q, items, ws)
        dplan = tc.tc_dequant_fp8_prepare(q, y, ditems, ws)
        assert plan.tiled == want_tiled and dplan.tiled == want_tiled and plan.full_tiles == 8
        _cast_and_check(src, bits, items, mats, q_off, s_off, ws_bytes)
        # the inverse of the oracle's codes, planned in the same workspace
        hq = np.zeros(q_off, dtype=np.uint8)
        hs = np.zeros(s_off, dtype=np.float32)
        for k, (so, rows, cols, ld) in enumerate(mats):
            view = np.lib.stride_tricks.as_strided(bits[so:], shape=(rows, cols), strides=(2 * ld, 2))
            cq, cs = oracle.cast_fp8_blockscaled(view)
            hq[int(items[k]["dst_off"]):int(items[k]["dst_off"]) + rows * cols] = cq.reshape(-1)
            hs[int(items[k]["scale_off"]):int(items[k]["scale_off"]) + cs.size] = cs.reshape(-1)
        qd = torch.from_numpy(hq).to(DEV)
        sd = torch.from_numpy(hs).to(DEV)
        dplan = tc.tc_dequant_fp8_prepare(qd, y, ditems, ws)
        assert dplan.tiled == want_tiled
        y.zero_()
        tc.tc_dequant_fp8_planned(qd, sd, y, ws, dplan)
        torch.cuda.synchronize()
        hy = _host(y.view(torch.int16)).view(np.uint16)
        for k, (so, rows, cols, ld) in enumerate(mats):
            o, tr, tcn = int(items[k]["dst_off"]), (rows + 127) // 128, (cols + 127) // 128
            cq = hq[o:o + rows * cols].reshape(rows, cols)
            cs = hs[int(items[k]["scale_off"]):int(items[k]["scale_off"]) + tr * tcn].reshape(tr, tcn)
            assert np.array_equal(hy[o:o + rows * cols].reshape(rows, cols),
                                  oracle.dequant_fp8_blockscaled(cq, cs)), (ws_bytes, k)


def test_blockscaled_special_tiles():
    rng = np.random.default_rng(53)
    a = rng.normal(0, 1, size=(256, 640)).astype(np.float32)
    a[0:128, 0:128] = 0.0
    a[0:128, 0:128][::3, ::5] = -0.0
    a[0:128, 128:256][7, 9] = np.inf
    a[0:128, 256:384][100, 1] = np.nan
    a[0:128, 384:512][3, 3] = -np.inf
    a[128:256, 0:128] *= 1e-38                  # subnormal bf16 values, subnormal scale
    a[128:256, 128:256] = 0.0
    a[128:256, 128:256][5, 5] = 2.0 ** -133
    a[128:256, 128:256][6, 6] = -(2.0 ** -133)
    a[128:256, 256:384] *= 1e30                 # huge values
    a[128:256, 384:512] = 448.0                 # amax exactly 448 -> scale 1
    a[128:256, 384:512][::2] = -1.0
    a[128:256, 512:640] = rng.choice([1.0, -2.0, 0.5, 3.0], size=(128, 128))  # exact quotients, ties
    bits = _bits_from_float(a).reshape(-1)
    _cast_matrices(bits, [(0, 256, 640, 640)])
    _cast_matrices(bits, [(1, 255, 600, 640)])  # the same through the edge path


def test_blockscaled_rounding_midpoints():
    """Tiles whose quotients land on and around E4M3 rounding midpoints."""
    rng = np.random.default_rng(54)
    mats = []
    parts = []
    off = 0
    for t in range(24):
        amax = float(np.float32(rng.uniform(0.5, 4.0)))
        s = np.float32(amax) / np.float32(448.0)
        # midpoints of the E4M3 grid, mapped back to x = mid * s, rounded to bf16
        mids = np.array([(a + b) / 2 for a, b in zip(_E4M3_POS[:-1], _E4M3_POS[1:])], dtype=np.float64)
        x = rng.choice(mids, size=128 * 128) * float(s) * rng.choice([-1.0, 1.0], size=128 * 128)
        x *= 1 + rng.integers(-4, 5, size=x.size) * 2.0 ** -9
        x[0] = amax
        bits = _bits_from_float(x.astype(np.float32))
        parts.append(bits)
        mats.append((off, 128, 128, 128))
        off += bits.size
    _cast_matrices(np.concatenate(parts), mats)


_E4M3_POS = sorted({abs(oracle.e4m3_decode(c)) for c in range(0x7F)})


def _tiles_under_amax(a_lo, a_hi):
    """For every tile maximum A in [a_lo, a_hi): tiles whose element 0 is A
    and whose other elements run through every bf16 pattern with magnitude
    <= A, both signs (zero-padded), as one 128-row matrix."""
    per = 128 * 128 - 1
    blocks = []
    for a in range(a_lo, a_hi):
        mags = np.arange(a + 1, dtype=np.uint16)
        vals = np.concatenate([mags, mags | np.uint16(0x8000)])
        t = -(-vals.size // per)
        body = np.zeros(t * per, np.uint16)
        body[:vals.size] = vals
        tiles = np.empty((t, per + 1), np.uint16)
        tiles[:, 0] = a
        tiles[:, 1:] = body.reshape(t, per)
        blocks.append(tiles)
    tiles = np.concatenate(blocks)
    return np.ascontiguousarray(tiles.reshape(-1, 128, 128).transpose(1, 0, 2).reshape(128, -1))


@pytest.mark.parametrize("tiled", [False, True])
@pytest.mark.parametrize("part", range(4))
def test_blockscaled_exhaustive_amax_and_value(part, tiled):
    """Every finite positive tile maximum A (bf16 0x0001 .. 0x7F7F, in four
    parts) with every bf16 value |x| <= A of both signs: all pairs of element
    and tile scale that a finite, non-zero tile can present to the full-tile
    kernel (its quotient and its choice of fast or dividing path depend on
    nothing else).  Codes and scales against the oracle, in chunks; through
    the kernel that searches the items and through the one that reads the
    per-tile table."""
    bounds = [1, 0x3F80, 0x5A00, 0x6D00, 0x7F80]     # about equal work per part
    a0, a1 = bounds[part], bounds[part + 1]
    step = 512 if part == 0 else 128
    # room for the largest chunk's per-tile table, or the item table alone
    big = np.zeros(1, dtype=tc.CAST_ITEM_DTYPE)
    big[0] = (0, 128, 128 * 4096, 128 * 4096, 0, 128 * 4096, 0, 4096)
    ws = torch.empty(tc.tc_cast_fp8_workspace_tiles(big) if tiled else tc.tc_cast_fp8_workspace(1),
                     dtype=torch.uint8, device=DEV)
    checked = 0
    for lo in range(a0, a1, step):
        m = _tiles_under_amax(lo, min(a1, lo + step))
        rows, cols = m.shape
        assert cols // 128 <= 4096          # the tiled workspace holds this chunk's table
        items = np.zeros(1, dtype=tc.CAST_ITEM_DTYPE)
        items[0] = (0, rows, cols, cols, 0, cols, 0, cols // 128)
        src = _to_dev_bits(m.reshape(-1))
        q = torch.empty(rows * cols, dtype=torch.uint8, device=DEV)
        sc = torch.empty(cols // 128, dtype=torch.float32, device=DEV)
        tc.tc_cast_fp8_blockscaled(src, q, sc, items, ws)
        torch.cuda.synchronize()
        want_q, want_s = oracle.cast_fp8_blockscaled(m)
        assert np.array_equal(_host(sc).view(np.uint32), want_s.reshape(-1).view(np.uint32)), lo
        got = _host(q).reshape(rows, cols)
        if not np.array_equal(got, want_q):
            r, c = np.argwhere(got != want_q)[0]
            raise AssertionError(f"A in [{lo}, {lo + step}): x={hex(int(m[r, c]))} gpu={hex(int(got[r, c]))} "
                                 f"oracle={hex(int(want_q[r, c]))}")
        checked += m.size
        del src, q, sc
    # every (A, x) pair of the part was cast: sum over A of 2 (A + 1) values
    assert checked >= sum(2 * (a + 1) for a in range(a0, a1))
    print(f"A in [{a0:#x}, {a1:#x}): {checked / 1e6:.0f} M elements checked")


@pytest.mark.parametrize("layers,ranks", [(2, [0, 7]), (10, [3])])
def test_tp_shard_cast_70b_layers(layers, ranks):
    """70B-shaped layers (hidden 8192, 64 q / 8 kv heads, MLP 28672), N(0, 0.02),
    cast into TP=8 shards, compared in full with the oracle.  Ten layers make
    70 items, so the kernel's item search takes its second round."""
    spec = synth.spec_70b(layers)
    n = synth.spec_elems(spec)
    stream = synth.bf16_normal(n, 0.02, synth.SEED_CAST_70B, device=DEV)
    host = _host(stream.view(torch.int16)).view(np.uint16)
    tp = 8
    for rank in ranks:
        items = tcv.cast_items(spec, tp, rank)
        q = torch.empty(tcv.shard_elems(spec, tp), dtype=torch.uint8, device=DEV)
        s = torch.empty(tcv.scale_elems(spec, tp), dtype=torch.float32, device=DEV)
        ws = torch.empty(tc.tc_cast_fp8_workspace(len(items)), dtype=torch.uint8, device=DEV)
        tc.tc_cast_fp8_blockscaled(stream, q, s, items, ws)
        torch.cuda.synchronize()
        hq, hs = _host(q), _host(s)
        off = 0
        for it, (_, rows, cols, split) in zip(items, spec):
            w = host[off:off + rows * cols].reshape(rows, cols)
            off += rows * cols
            want_q, want_s = oracle.cast_fp8_blockscaled(oracle.tp_slice(w, split, tp, rank))
            r, c = want_q.shape
            assert np.array_equal(hq[it["dst_off"]:it["dst_off"] + r * c].reshape(r, c), want_q)
            tr, tcn = want_s.shape
            got_s = hs[it["scale_off"]:it["scale_off"] + tr * tcn].reshape(tr, tcn)
            assert np.array_equal(got_s.view(np.uint32), want_s.view(np.uint32))
    del stream
    torch.cuda.empty_cache()


def _sampled_tiles_match_oracle(src, q, s, items, rng, count):
    """count random 128x128 tiles of random items: codes and scale bits of
    the GPU cast against the oracle's cast of the same source tile."""
    for k in rng.choice(len(items), size=min(count, len(items)), replace=False):
        it = items[k]
        rows, cols = int(it["rows"]), int(it["cols"])
        tr, tcn = (rows + 127) // 128, (cols + 127) // 128
        ti, tj = int(rng.integers(0, tr)), int(rng.integers(0, tcn))
        r0, c0 = ti * 128, tj * 128
        ld = int(it["src_ld"])
        base = int(it["src_off"]) + r0 * ld + c0
        tile = _host(src[base:base + 127 * ld + 128].view(torch.int16)).view(np.uint16)
        view = np.lib.stride_tricks.as_strided(tile, shape=(128, 128), strides=(2 * ld, 2))
        want_q, want_s = oracle.cast_fp8_blockscaled(view)
        dld = int(it["dst_ld"])
        dq = int(it["dst_off"]) + r0 * dld + c0
        got_q = _host(q[dq:dq + 127 * dld + 128])
        got_q = np.lib.stride_tricks.as_strided(got_q, shape=(128, 128), strides=(dld, 1))
        assert np.array_equal(got_q, want_q), (k, ti, tj)
        got_s = _host(s[int(it["scale_off"]) + ti * int(it["scale_ld"]) + tj])
        assert got_s.view(np.uint32) == want_s.view(np.uint32)[0, 0]


def _item_matches_oracle(src, q, hs, it):
    """One cast item in full: the oracle's cast of a host copy of the item's
    (strided) source rows against the GPU's codes and scale grid."""
    rows, cols, ld = int(it["rows"]), int(it["cols"]), int(it["src_ld"])
    so = int(it["src_off"])
    x = src[so:so + (rows - 1) * ld + cols].as_strided((rows, cols), (ld, 1)).contiguous()
    hx = _host(x.view(torch.int16)).view(np.uint16)
    want_q, want_s = oracle.cast_fp8_blockscaled(hx)
    dld, do = int(it["dst_ld"]), int(it["dst_off"])
    got_q = q[do:do + (rows - 1) * dld + cols].as_strided((rows, cols), (dld, 1)).contiguous()
    assert np.array_equal(_host(got_q), want_q), it
    tr, tcn = want_s.shape
    sld, sof = int(it["scale_ld"]), int(it["scale_off"])
    got_s = np.lib.stride_tricks.as_strided(hs[sof:], shape=(tr, tcn), strides=(4 * sld, 4))
    assert np.array_equal(got_s.view(np.uint32), want_s.view(np.uint32)), it


def _every_tile_reaches_448(q, items):
    """The element with |x| = amax encodes to +-448 (0x7E / 0xFE): the
    largest code magnitude of every tile is 0x7E.  Item sizes here are
    multiples of 128."""
    for it in items:
        rows, cols, ld, off = int(it["rows"]), int(it["cols"]), int(it["dst_ld"]), int(it["dst_off"])
        assert rows % 128 == 0 and cols % 128 == 0
        m = q[off:off + (rows - 1) * ld + cols].as_strided((rows, cols), (ld, 1))
        mag = torch.bitwise_and(m, 0x7F).contiguous().view(rows // 128, 128, cols // 128, 128)
        tmax = mag.amax(dim=(1, 3))
        assert bool((tmax == 0x7E).all()), int(tmax.min())


def test_tp_shard_cast_70b_full_size():
    """All 80 layers (136.9 GB of bf16 in HBM), rank 3 of TP=8: the shard
    slices hold N(0, 0.02) values and everything outside them is poisoned with
    a huge value, so a read outside the slice would change the scales.
    Every item against the oracle, codes and scale bits; every scale is
    checked to be a normal N(0, 0.02) tile scale (no poison), and every tile's
    largest code is +-448.
    Then the inverse rule over the whole shard: every item against the
    oracle's inverse of the GPU codes, and every element within the E4M3 +
    bf16 rounding bound of its source value."""
    tp, rank = 8, 3
    spec = synth.spec_70b(80)
    n = synth.spec_elems(spec)
    stream = torch.full((n,), 3.0e38, dtype=torch.bfloat16, device=DEV)
    items = tcv.cast_items(spec, tp, rank)
    fill = synth.bf16_normal(tcv.shard_elems(spec, tp), 0.02, synth.SEED_CAST_70B, device=DEV)
    # place the values into the rank's slices with torch indexing
    off = 0
    foff = 0
    for (_, rows, cols, split) in spec:
        w = stream[off:off + rows * cols].view(rows, cols)
        off += rows * cols
        sl = w[rank * rows // tp:(rank + 1) * rows // tp] if split == "rows" else \
            w[:, rank * cols // tp:(rank + 1) * cols // tp]
        k = sl.numel()
        sl.copy_(fill[foff:foff + k].view(sl.shape))
        foff += k
    del fill
    q = torch.empty(tcv.shard_elems(spec, tp), dtype=torch.uint8, device=DEV)
    s = torch.empty(tcv.scale_elems(spec, tp), dtype=torch.float32, device=DEV)
    # the timed configuration: a workspace with the per-tile table
    ws = torch.empty(tc.tc_cast_fp8_workspace_tiles(items), dtype=torch.uint8, device=DEV)
    plan = tc.tc_cast_fp8_prepare(stream, q, items, ws)
    assert plan.tiled == 1 and plan.full_tiles == tcv.scale_elems(spec, tp)
    tc.tc_cast_fp8_planned(stream, q, s, ws, plan)
    torch.cuda.synchronize()
    # no poisoned tile: every scale is what an N(0, 0.02) tile gives
    assert bool(((s > 1e-5) & (s < 1e-3)).all())
    _every_tile_reaches_448(q, items)
    # every item against the oracle, layer by layer (80 passes over host
    # copies of the items' strided source rows)
    hs = _host(s)
    for k, it in enumerate(items):
        if k % 70 == 0:
            print(f"cast item {k} of {len(items)}", flush=True)
        _item_matches_oracle(stream, q, hs, it)

    # the inverse rule over the whole shard
    ditems = tcv.dequant_items(spec, tp)
    y = torch.empty(tcv.shard_elems(spec, tp), dtype=torch.bfloat16, device=DEV)
    dws = torch.empty(tc.tc_dequant_fp8_workspace_tiles(ditems), dtype=torch.uint8, device=DEV)
    dplan = tc.tc_dequant_fp8_prepare(q, y, ditems, dws)
    assert dplan.tiled == 1
    tc.tc_dequant_fp8_planned(q, s, y, dws, dplan)
    torch.cuda.synchronize()
    smax = float(s.max())
    for it, dit in zip(items, ditems):
        rows, cols = int(it["rows"]), int(it["cols"])
        x = stream[int(it["src_off"]):int(it["src_off"]) + (rows - 1) * int(it["src_ld"]) + cols]
        x = x.as_strided((rows, cols), (int(it["src_ld"]), 1)).float()
        yy = y[int(dit["dst_off"]):int(dit["dst_off"]) + rows * cols].view(rows, cols).float()
        # E4M3 keeps 3 mantissa bits (half an ulp: 2^-4 relative), bf16 adds
        # 2^-8; below the normal range the step is s * 2^-9 (half: s * 2^-10)
        bound = (2.0 ** -4 + 2.0 ** -8 + 2.0 ** -12) * x.abs() + smax * 2.0 ** -10
        assert bool(((yy - x).abs() <= bound).all()), it
    # every item of the inverse against the oracle's inverse of the GPU codes
    for k, dit in enumerate(ditems):
        if k % 70 == 0:
            print(f"inverse item {k} of {len(ditems)}", flush=True)
        rows, cols = int(dit["rows"]), int(dit["cols"])
        assert int(dit["src_ld"]) == cols and int(dit["dst_ld"]) == cols
        qo, yo = int(dit["src_off"]), int(dit["dst_off"])
        qt = _host(q[qo:qo + rows * cols]).reshape(rows, cols)
        tr, tcn = (rows + 127) // 128, (cols + 127) // 128
        so = int(dit["scale_off"])
        st = hs[so:so + tr * tcn].reshape(tr, tcn)
        want = oracle.dequant_fp8_blockscaled(qt, st)
        got = _host(y[yo:yo + rows * cols].view(torch.int16)).view(np.uint16).reshape(rows, cols)
        assert np.array_equal(got, want), k
    del stream, q, s, y
    torch.cuda.empty_cache()


def test_reshard_cast_70b_full_size():
    """The timed reshard into fp8 at full size: 70B-shaped weights held as the
    eight bf16 shards of a TP=8 split (136.9 GB, N(0, 0.02)) cast into rank 1
    of a TP=4 split.  Every item against the oracle; every scale in the
    N(0, 0.02) range; every tile's largest code is +-448."""
    src_tp, dst_tp, rank = 8, 4, 1
    spec = synth.spec_70b(80)
    n = synth.spec_elems(spec)
    src = synth.bf16_normal(n, 0.02, synth.SEED_CAST_70B, device=DEV)
    items = tcv.reshard_cast_items(spec, src_tp, dst_tp, rank)
    q = torch.empty(tcv.shard_elems(spec, dst_tp), dtype=torch.uint8, device=DEV)
    s = torch.full((tcv.scale_elems(spec, dst_tp),), float("nan"), dtype=torch.float32, device=DEV)
    ws = torch.empty(tc.tc_cast_fp8_workspace_tiles(items), dtype=torch.uint8, device=DEV)
    tc.tc_cast_fp8_blockscaled(src, q, s, items, ws)
    torch.cuda.synchronize()
    assert bool(((s > 1e-5) & (s < 1e-3)).all())      # every scale written, none poisoned
    _every_tile_reaches_448(q, items)
    hs = _host(s)
    for k, it in enumerate(items):
        if k % 140 == 0:
            print(f"reshard-cast item {k} of {len(items)}", flush=True)
        _item_matches_oracle(src, q, hs, it)
    del src, q, s
    torch.cuda.empty_cache()


# ---------------------------------------------------------------------------
# inverse cast
# ---------------------------------------------------------------------------

def _dequant_matrices(codes_1d: np.ndarray, scales_1d: np.ndarray, mats, dst_pad=0):
    """mats: (code_off, rows, cols, code_ld, scale_off, scale_ld); bf16 outputs
    packed with row stride cols + dst_pad.  Compared with the oracle."""
    items = np.zeros(len(mats), dtype=tc.DEQUANT_ITEM_DTYPE)
    y_off = 0
    for k, (qo, rows, cols, ld, so, sld) in enumerate(mats):
        items[k] = (qo, rows, cols, ld, y_off, cols + dst_pad, so, sld)
        y_off += rows * (cols + dst_pad)
    q = torch.from_numpy(codes_1d).to(DEV)
    s = torch.from_numpy(scales_1d.astype(np.float32)).to(DEV)
    # the item table alone, then with the per-tile table as well
    for ws_bytes in (tc.tc_dequant_fp8_workspace(len(mats)), tc.tc_dequant_fp8_workspace_tiles(items)):
        _dequant_and_check(codes_1d, scales_1d, mats, items, q, s, y_off, ws_bytes)


def _dequant_and_check(codes_1d, scales_1d, mats, items, q, s, y_off, ws_bytes):
    y = torch.full((max(y_off, 1),), -1, dtype=torch.int16, device=DEV)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
    tc.tc_dequant_fp8_blockscaled(q, s, y, items, ws)
    torch.cuda.synchronize()
    hy = _host(y).view(np.uint16)
    for k, (qo, rows, cols, ld, so, sld) in enumerate(mats):
        it = items[k]
        qv = np.lib.stride_tricks.as_strided(codes_1d[qo:], shape=(rows, cols), strides=(ld, 1))
        tr, tcn = (rows + 127) // 128, (cols + 127) // 128
        sv = np.lib.stride_tricks.as_strided(scales_1d.astype(np.float32)[so:], shape=(tr, tcn),
                                             strides=(4 * sld, 4))
        want = oracle.dequant_fp8_blockscaled(qv, np.ascontiguousarray(sv))
        got = np.lib.stride_tricks.as_strided(hy[int(it["dst_off"]):], shape=(rows, cols),
                                              strides=(2 * int(it["dst_ld"]), 2))
        if not np.array_equal(got, want):
            bad = np.argwhere(got != want)
            r, c = bad[0]
            raise AssertionError(f"matrix {k}: {len(bad)} differ, first {(r, c)}: q={hex(int(qv[r, c]))} "
                                 f"gpu={hex(int(got[r, c]))} oracle={hex(int(want[r, c]))}")


def test_dequant_every_code_many_scales():
    rng = np.random.default_rng(70)
    sbits = np.concatenate([rng.integers(0x00800000, 0x7F000000, size=40, dtype=np.int64),
                            rng.integers(1, 0x00800000, size=6, dtype=np.int64),
                            [0, 0x80000000, 0x3F800000, 0x7F7FFFFF, 0x7F800000, 0x7FC00000]]).astype(np.uint32)
    scales = sbits.view(np.float32)
    codes = np.tile(np.arange(256, dtype=np.uint8), 128 * 2).reshape(-1)        # [128][512]
    mats = [(0, 128, 512, 512, 4 * k, 4) for k in range(len(scales))]          # one scale per tile row
    sgrid = np.repeat(scales, 4)
    _dequant_matrices(codes, sgrid, mats)


@pytest.mark.parametrize("part", range(4))
def test_dequant_every_code_at_every_cast_scale(part):
    """Every E4M3 code at every scale a cast can produce for a finite,
    non-zero tile, s = RN_f32(A / 448) for bf16 A = 0x0001 .. 0x7F7F (in four
    parts): one full 128x128 tile per scale holding each code 64 times,
    through the full-tile kernel, against the oracle."""
    a = np.arange(1, 0x7F80, dtype=np.uint32)
    a = np.array_split(a, 4)[part]
    scales = (a << np.uint32(16)).view(np.float32) / np.float32(448.0)   # IEEE single division
    tile = np.tile(np.arange(256, dtype=np.uint8), 64).reshape(128, 128)
    for chunk in np.array_split(scales, 8):
        t = len(chunk)
        codes = np.ascontiguousarray(np.broadcast_to(tile, (t, 128, 128)).transpose(1, 0, 2)).reshape(-1)
        _dequant_matrices(codes, chunk, [(0, 128, 128 * t, 128 * t, 0, t)])


def test_dequant_ragged_strided_unaligned():
    rng = np.random.default_rng(71)
    codes = rng.integers(0, 256, size=700 * 600, dtype=np.int64).astype(np.uint8)
    scales = (rng.uniform(0.5, 2, size=64) * 10.0 ** rng.integers(-20, 20, size=64)).astype(np.float32)
    scales[5] = 0.0
    scales[9] = np.nan
    mats = [(0, 256, 384, 384, 0, 3),        # whole tiles
            (0, 300, 200, 600, 10, 2),       # ragged, strided
            (8, 128, 128, 600, 20, 1),       # aligned strided tile
            (3, 130, 129, 600, 30, 2),       # unaligned codes
            (1000, 1, 1, 1, 40, 1),
            (2000, 5, 300, 301, 50, 3)]
    _dequant_matrices(codes, scales, mats)
    _dequant_matrices(codes, scales, mats, dst_pad=3)   # unaligned bf16 rows


@pytest.mark.parametrize("tiled", [False, True])
def test_cast_then_dequant_70b_layers(tiled):
    """Ten 70B-shaped layers (70 items: the item search's second round): cast
    rank 5 of TP=8 to fp8, dequantize the shard back to bf16, and compare both
    results with the oracle in full; with the item table alone and with the
    per-tile table."""
    spec = synth.spec_70b(10)
    n = synth.spec_elems(spec)
    stream = synth.bf16_normal(n, 0.02, synth.SEED_CAST_70B, device=DEV)
    tp, rank = 8, 5
    items = tcv.cast_items(spec, tp, rank)
    q = torch.empty(tcv.shard_elems(spec, tp), dtype=torch.uint8, device=DEV)
    s = torch.empty(tcv.scale_elems(spec, tp), dtype=torch.float32, device=DEV)
    ws = torch.empty(tc.tc_cast_fp8_workspace_tiles(items) if tiled else tc.tc_cast_fp8_workspace(len(items)),
                     dtype=torch.uint8, device=DEV)
    tc.tc_cast_fp8_blockscaled(stream, q, s, items, ws)
    y = torch.empty(tcv.shard_elems(spec, tp), dtype=torch.bfloat16, device=DEV)
    ditems = tcv.dequant_items(spec, tp)
    dws = torch.empty(tc.tc_dequant_fp8_workspace_tiles(ditems) if tiled else
                      tc.tc_dequant_fp8_workspace(len(ditems)), dtype=torch.uint8, device=DEV)
    tc.tc_dequant_fp8_blockscaled(q, s, y, ditems, dws)
    torch.cuda.synchronize()
    hq, hs, hy = _host(q), _host(s), _host(y.view(torch.int16)).view(np.uint16)
    host = _host(stream.view(torch.int16)).view(np.uint16)
    off = 0
    for it, dit, (_, rows, cols, split) in zip(items, ditems, spec):
        w = host[off:off + rows * cols].reshape(rows, cols)
        off += rows * cols
        want_q, want_s = oracle.cast_fp8_blockscaled(oracle.tp_slice(w, split, tp, rank))
        r, c = want_q.shape
        assert np.array_equal(hq[it["dst_off"]:it["dst_off"] + r * c].reshape(r, c), want_q)
        want_y = oracle.dequant_fp8_blockscaled(want_q, want_s)
        assert np.array_equal(hy[dit["dst_off"]:dit["dst_off"] + r * c].reshape(r, c), want_y)
    del stream
    torch.cuda.empty_cache()


def _torch_shards(stream, spec, tp):
    """All tp shards of a contiguous stream, rank-major (torch slicing on the device)."""
    parts = []
    for r in range(tp):
        off = 0
        for (_, rows, cols, split) in spec:
            w = stream[off:off + rows * cols].view(rows, cols)
            off += rows * cols
            sl = w[r * rows // tp:(r + 1) * rows // tp] if split == "rows" else \
                w[:, r * cols // tp:(r + 1) * cols // tp]
            parts.append(sl.reshape(-1))
    return torch.cat(parts)


@pytest.mark.parametrize("src_tp,dst_tp,ranks", [(8, 4, [1, 2]), (4, 8, [5]), (8, 1, [0])])
def test_reshard_cast_70b_layers(src_tp, dst_tp, ranks):
    """Two 70B-shaped layers held as src_tp bf16 shards, cast straight into
    rank r of a dst_tp fp8 split: every code and scale equals the oracle's cast
    of that rank's slices of the full weights."""
    spec = synth.spec_70b(2)
    n = synth.spec_elems(spec)
    stream = synth.bf16_normal(n, 0.02, synth.SEED_CAST_70B, device=DEV)
    host = _host(stream.view(torch.int16)).view(np.uint16)
    src = _torch_shards(stream, spec, src_tp)
    del stream
    for rank in ranks:
        items = tcv.reshard_cast_items(spec, src_tp, dst_tp, rank)
        q = torch.empty(tcv.shard_elems(spec, dst_tp), dtype=torch.uint8, device=DEV)
        s = torch.empty(tcv.scale_elems(spec, dst_tp), dtype=torch.float32, device=DEV)
        ws = torch.empty(tc.tc_cast_fp8_workspace(len(items)), dtype=torch.uint8, device=DEV)
        tc.tc_cast_fp8_blockscaled(src, q, s, items, ws)
        torch.cuda.synchronize()
        hq, hs = _host(q), _host(s).view(np.uint32)
        qoffs, _ = tcv.shard_slice_offsets(spec, dst_tp, 1)
        soffs = tcv.scale_offsets(spec, dst_tp)
        off = 0
        for k, (_, rows, cols, split) in enumerate(spec):
            w = host[off:off + rows * cols].reshape(rows, cols)
            off += rows * cols
            want_q, want_s = oracle.cast_fp8_blockscaled(oracle.tp_slice(w, split, dst_tp, rank))
            r, c = want_q.shape
            assert np.array_equal(hq[qoffs[k]:qoffs[k] + r * c].reshape(r, c), want_q), (k, rank)
            tr, tcn = want_s.shape
            assert np.array_equal(hs[soffs[k]:soffs[k] + tr * tcn].reshape(tr, tcn),
                                  want_s.view(np.uint32)), (k, rank)
    del src
    torch.cuda.empty_cache()
