"""GPU parity on seeded random inputs, each case against the oracle.

* Fragment lists of mixed lengths (empty, tiny, log-uniform, large), at byte
  and 16-byte alignment, from one fragment up to lists long enough to be
  planned in destination order; planned with the recommended and with the
  smallest workspace (larger pieces); copied with and without digests, and
  digested again from the destination.
* Ragged cast items (random shapes, row strides, element offsets, code and
  scale padding) over values of random magnitude with zeros, subnormals and
  now and then an Inf or NaN; the codes are then decoded by the inverse.
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
    torch.cuda.synchronize()
    hsrc = _host(src)
    want = np.full(dp, 0x5A, dtype=np.uint8)
    oracle.copy_fragments(hsrc, want, frags)
    got = _host(dst)
    assert np.array_equal(got, want), f"{int((got != want).sum())} bytes differ"
    assert np.array_equal(_host(again), want)
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
