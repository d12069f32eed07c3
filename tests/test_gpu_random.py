"""GPU parity on seeded random inputs, each case against the oracle.

* Fragment lists of mixed lengths (empty, tiny, log-uniform, large), at byte
  and 16-byte alignment, from one fragment up to lists long enough to be
  planned in destination order; planned with the recommended and with the
  smallest workspace (larger pieces); copied with and without digests, and
  digested again from the destination.
* Ragged cast items (random shapes, row strides, element offsets, code and
  scale padding) over values of random magnitude with zeros, subnormals and
  now and then an Inf or NaN; the codes are then decoded by the inverse.
* Random block pools (region count, block size, stride, unaligned region
  bases, repeated ids) through gather and scatter, and random staging rings
  through publish and hydrate.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_06007_amd as tc
from tests.test_gpu_cast import _bits_from_float, _cast_matrices, _dequant_matrices

pytestmark = pytest.mark.gpu

DEV = "cuda:0"

# (seed, fragments, alignment, smallest workspace)
FRAG_CASES = [(0, 1, 16, False), (1, 2, 1, False), (2, 7, 16, True), (3, 100, 1, False),
              (4, 1000, 16, False), (5, 1000, 1, True), (6, 4095, 16, False), (7, 4096, 16, False),
              (8, 4096, 1, False), (9, 5000, 16, True), (10, 12000, 16, False), (11, 12000, 1, False),
              (12, 20000, 16, True), (13, 3, 1, True), (14, 333, 16, False), (15, 8191, 1, True)]


def _host(t):
    return t.detach().to("cpu").numpy()


@pytest.mark.parametrize("seed,n,align,small_ws", FRAG_CASES)
def test_random_fragment_lists(seed, n, align, small_ws):
    frags, sp, dp = synth.fragment_mix(n, 900 + seed, align=align, big_max=512 * 1024)
    print(f"case seed={seed} n={n} align={align} small_ws={small_ws} payload={int(frags[:, 2].sum())}",
          flush=True)
    src = synth.random_bytes(sp, 1900 + seed, device=DEV)
    dst = torch.full((dp,), 0x5A, dtype=torch.uint8, device=DEV)
    fr = torch.from_numpy(frags.view(np.int64)).to(DEV)
    ws_bytes = tc.tc_copy_fragments_workspace_min(n) if small_ws else tc.tc_copy_fragments_workspace(n)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
    total = tc.tc_plan_fragments(fr, ws)
    dg = torch.zeros(2 * n, dtype=torch.int64, device=DEV)
    tc.tc_copy_planned_digest(src, dst, ws, total, n, dg)
    dg_dst = torch.zeros_like(dg)
    tc.tc_digest_planned(dst, tc.DIGEST_DST, ws, total, n, dg_dst)
    again = torch.full_like(dst, 0x5A)
    tc.tc_copy_planned(src, again, ws, total)
    # the asynchronous one-call copy on a workspace of the same size: its plan
    # (piece, reordering) is decided on the device and the copy reads the count
    ws2 = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
    third = torch.full_like(dst, 0x5A)
    tc.tc_copy_fragments(src, third, fr, ws2)
    assert tc.tc_plan_status(ws2) == total
    torch.cuda.synchronize()
    hsrc = _host(src)
    want = np.full(dp, 0x5A, dtype=np.uint8)
    oracle.copy_fragments(hsrc, want, frags)
    got = _host(dst)
    assert np.array_equal(got, want), f"{int((got != want).sum())} bytes differ"
    assert np.array_equal(_host(again), want)
    assert np.array_equal(_host(third), want)
    wd = oracle.fragment_digests(hsrc, frags, use_src=True)
    assert np.array_equal(_host(dg).view(np.uint64).reshape(n, 2), wd)
    assert np.array_equal(_host(dg_dst).view(np.uint64).reshape(n, 2),
                          oracle.fragment_digests(want, frags, use_src=False))


def _random_values(rng, count):
    """bf16 bit patterns: normal values at a random magnitude, with zeros of
    both signs, subnormals, and rarely an Inf or a NaN."""
    mag = 10.0 ** rng.uniform(-30, 30)
    bits = _bits_from_float(rng.normal(0.0, mag, size=count).astype(np.float32))
    bits = bits.copy()
    pick = rng.random(count)
    bits[pick < 0.02] = 0x0000
    bits[(pick >= 0.02) & (pick < 0.03)] = 0x8000
    sub = (pick >= 0.03) & (pick < 0.04)
    bits[sub] = rng.integers(1, 0x80, size=int(sub.sum())).astype(np.uint16) | \
        (rng.integers(0, 2, size=int(sub.sum())).astype(np.uint16) << 15)
    if rng.random() < 0.3:
        bits[rng.integers(0, count)] = rng.choice([0x7F80, 0xFF80, 0x7FC1, 0xFFFF])
    return bits


@pytest.mark.parametrize("seed", range(12))
def test_random_cast_items_and_inverse(seed):
    rng = np.random.default_rng(3100 + seed)
    mats, off = [], int(rng.integers(0, 9))
    for _ in range(int(rng.integers(1, 6))):
        rows = int(128 * rng.integers(0, 3) + rng.choice([0, int(rng.integers(1, 128))]))
        cols = int(128 * rng.integers(0, 3) + rng.choice([0, int(rng.integers(1, 128))]))
        rows, cols = max(rows, 1), max(cols, 1)
        ld = cols + int(rng.choice([0, 0, 8, int(rng.integers(1, 40))]))
        mats.append((off, rows, cols, ld))
        off += (rows - 1) * ld + cols + int(rng.integers(0, 17))
    code_pad, scale_pad = int(rng.choice([0, 0, 8, 5])), int(rng.integers(0, 3))
    print(f"case seed={seed} mats={mats} code_pad={code_pad} scale_pad={scale_pad}", flush=True)
    bits = _random_values(rng, off + 16)
    _cast_matrices(bits, mats, code_pad=code_pad, scale_pad=scale_pad)
    # the inverse, in the same packed layout, on codes and scales that the
    # oracle's cast produced
    dmats, q_off, s_off, qs, ss = [], 0, 0, [], []
    for (so, rows, cols, ld) in mats:
        view = np.lib.stride_tricks.as_strided(bits[so:], shape=(rows, cols), strides=(2 * ld, 2))
        q, sc = oracle.cast_fp8_blockscaled(view)
        tr, tcn = sc.shape
        qs.append(np.pad(q, ((0, 0), (0, code_pad)), constant_values=0xCC).reshape(-1))
        ss.append(np.pad(sc, ((0, 0), (0, scale_pad)), constant_values=-7.0).reshape(-1))
        dmats.append((q_off, rows, cols, cols + code_pad, s_off, tcn + scale_pad))
        q_off += rows * (cols + code_pad)
        s_off += tr * (tcn + scale_pad)
    codes = np.concatenate(qs).astype(np.uint8)
    scales = np.concatenate(ss).astype(np.float32)
    _dequant_matrices(codes, scales, dmats, dst_pad=int(rng.choice([0, 3])))


@pytest.mark.parametrize("seed", range(12))
def test_random_block_pools(seed):
    """Random pools: 1-8 regions, block sizes from 1 byte to 70,000 (16-byte
    multiples half the time), stride pads, region bases at random byte
    offsets inside one allocation, ids with repeats for the gather and
    distinct for the scatter."""
    rng = np.random.default_rng(4100 + seed)
    R = int(rng.integers(1, 9))
    B = int(rng.integers(1, 70000))
    if rng.random() < 0.5:
        B = max(16, (B // 16) * 16)
    stride = B + int(rng.choice([0, 16, int(rng.integers(1, 64))]))
    nb = int(rng.integers(1, 200))
    n = int(rng.integers(1, 3 * nb + 1))
    span = (nb - 1) * stride + B
    lead = [int(rng.choice([0, 16, int(rng.integers(0, 64))])) for _ in range(R)]
    print(f"case seed={seed} R={R} B={B} stride={stride} nb={nb} n={n} lead={lead}", flush=True)
    whole = synth.random_bytes(sum(lead) + R * span, 5100 + seed, device=DEV)
    regions, pos = [], 0
    for r in range(R):
        pos += lead[r]
        regions.append(whole[pos:pos + span])
        pos += span
    ids_np = rng.integers(0, nb, size=n).astype(np.int32)           # repeats allowed
    ids = torch.from_numpy(ids_np).to(DEV)
    out = torch.empty(n * R * B, dtype=torch.uint8, device=DEV)
    tc.tc_gather_blocks(regions, nb, B, stride, ids, out)
    uniq_np = rng.permutation(nb)[:int(rng.integers(1, nb + 1))].astype(np.int32)
    uniq = torch.from_numpy(uniq_np).to(DEV)
    inp = synth.random_bytes(len(uniq_np) * R * B, 6100 + seed, device=DEV)
    dst_whole = torch.full_like(whole, 0x3C)
    dst = []
    pos = 0
    for r in range(R):
        pos += lead[r]
        dst.append(dst_whole[pos:pos + span])
        pos += span
    tc.tc_scatter_blocks(dst, nb, B, stride, uniq, inp)
    torch.cuda.synchronize()
    hosts = [_host(x) for x in regions]
    want = oracle.gather_blocks(hosts, B, stride, ids_np)
    assert np.array_equal(_host(out).reshape(want.shape), want)
    back = [np.full(span, 0x3C, np.uint8) for _ in range(R)]
    oracle.scatter_blocks(back, B, stride, uniq_np, _host(inp).reshape(len(uniq_np), R, B))
    hd = _host(dst_whole)
    pos = 0
    for r in range(R):
        assert np.all(hd[pos:pos + lead[r]] == 0x3C)            # the gaps between regions
        pos += lead[r]
        assert np.array_equal(hd[pos:pos + span], back[r]), f"region {r}"
        pos += span
    assert np.all(hd[pos:] == 0x3C)


@pytest.mark.parametrize("seed", range(6))
def test_random_staging(seed):
    """Random rings (2-6 slots of 4 KiB to 1 MiB, 1-4 host threads) moving a
    random number of ids through publish and hydrate, pageable or pinned."""
    rng = np.random.default_rng(7100 + seed)
    R, B = int(rng.integers(1, 5)), int(rng.choice([4096, 4096 + 16, 512, 100]))
    nb = int(rng.integers(20, 300))
    per_id = R * B
    slot = int(max(per_id, rng.integers(4096, 1 << 20)))
    slots, threads = int(rng.integers(2, 7)), int(rng.integers(1, 5))
    pinned = bool(rng.random() < 0.5)
    n = int(rng.integers(1, nb + 1))
    print(f"case seed={seed} R={R} B={B} nb={nb} n={n} slot={slot} slots={slots} threads={threads} "
          f"pinned={pinned}", flush=True)
    span = nb * B
    regions = [synth.random_bytes(span, 8100 + seed * 8 + r, device=DEV) for r in range(R)]
    ids_np = rng.permutation(nb)[:n].astype(np.int32)
    ids = torch.from_numpy(ids_np).to(DEV)
    stage = torch.empty(int(rng.integers(1, 4)) * slot, dtype=torch.uint8, device=DEV)
    if pinned:
        host = torch.zeros(n * per_id, dtype=torch.uint8).pin_memory()
    else:
        host = np.zeros(n * per_id, dtype=np.uint8)
    with tc.Stager(slot_bytes=slot, slots=slots, host_threads=threads) as st:
        tc.tc_publish_to_host(st.handle, regions, nb, B, B, ids, host, stage)
        hb = host.numpy() if pinned else host
        hosts = [_host(r) for r in regions]
        want = oracle.gather_blocks(hosts, B, B, ids_np)
        assert np.array_equal(hb.reshape(want.shape), want)
        dst = [torch.full_like(r, 0x77) for r in regions]
        tc.tc_hydrate_from_host(st.handle, dst, nb, B, B, ids, host, stage)
        torch.cuda.synchronize()
    back = [np.full(span, 0x77, np.uint8) for _ in range(R)]
    oracle.scatter_blocks(back, B, B, ids_np, want)
    for r in range(R):
        assert np.array_equal(_host(dst[r]), back[r]), f"region {r}"
