"""Pins for the oracle's byte movers and tensor-parallel slicing (CPU only).

Checked against library routines (torch.index_select, numpy fancy
indexing, torch.chunk / torch.cat) and properties that fix the result:
round trips, untouched sentinel bytes, order independence, permutation
inverses, conservation of bytes.
"""
import numpy as np
import pytest
import torch

import oracle
import synth


def _pool(R, nb, B, stride, seed):
    rng = np.random.default_rng(seed)
    return [rng.integers(0, 256, size=(nb - 1) * stride + B, dtype=np.uint8) for _ in range(R)]


@pytest.mark.parametrize("stride_pad", [0, 48])
def test_gather_matches_index_select_and_address_formula(stride_pad):
    R, nb, B = 4, 64, 96
    stride = B + stride_pad
    regions = _pool(R, nb, B, stride, 1)
    ids = synth.ids_without_replacement(nb, 20, seed=2)
    out = oracle.gather_blocks(regions, B, stride, ids)
    # per-byte address formula with numpy fancy indexing
    for r in range(R):
        idx = ids[:, None].astype(np.int64) * stride + np.arange(B)[None, :]
        assert np.array_equal(out[:, r, :], regions[r][idx])
    # torch.index_select on a [num_blocks, stride] view (library routine)
    if stride_pad == 0:
        for r in range(R):
            t = torch.from_numpy(regions[r]).view(nb, B)
            ref = torch.index_select(t, 0, torch.from_numpy(ids.astype(np.int64)))
            assert np.array_equal(out[:, r, :], ref.numpy())


def test_gather_allows_repeated_ids_and_rejects_out_of_range():
    R, nb, B = 2, 8, 32
    regions = _pool(R, nb, B, B, 3)
    ids = np.array([3, 3, 0, 7], dtype=np.int32)
    out = oracle.gather_blocks(regions, B, B, ids)
    assert np.array_equal(out[0], out[1])
    with pytest.raises(ValueError):
        oracle.gather_blocks(regions, B, B, np.array([8], dtype=np.int32))
    with pytest.raises(ValueError):
        oracle.gather_blocks(regions, B, B, np.array([-1], dtype=np.int32))


def test_scatter_round_trips_and_leaves_other_blocks():
    R, nb, B, stride = 3, 50, 64, 80
    src = _pool(R, nb, B, stride, 4)
    ids = synth.ids_without_replacement(nb, 17, seed=5)
    buf = oracle.gather_blocks(src, B, stride, ids)
    dst = [np.full_like(r, 0xA5) for r in src]
    oracle.scatter_blocks(dst, B, stride, ids, buf)
    # gather after scatter gives the buffer back
    assert np.array_equal(oracle.gather_blocks(dst, B, stride, ids), buf)
    # every byte outside the written blocks is still the sentinel
    written = np.zeros(dst[0].size, dtype=bool)
    for i in ids:
        written[i * stride:i * stride + B] = True
    for r in range(R):
        assert np.all(dst[r][~written] == 0xA5)
        assert np.array_equal(dst[r][written], src[r][written])
    # scattering a pool's own blocks back leaves it unchanged
    before = [r.copy() for r in src]
    oracle.scatter_blocks(src, B, stride, ids, buf)
    for a, b in zip(src, before):
        assert np.array_equal(a, b)


def test_scatter_rejects_repeated_ids():
    R, nb, B = 1, 8, 16
    dst = _pool(R, nb, B, B, 6)
    with pytest.raises(ValueError):
        oracle.scatter_blocks(dst, B, B, np.array([1, 1], dtype=np.int32), np.zeros(2 * B, np.uint8))


@pytest.mark.parametrize("align", [16, 1])
def test_copy_fragments_properties(align):
    n, pool = 3000, 64 << 20
    frags = synth.fragment_storm(n, pool, seed=8, align=align)
    rng = np.random.default_rng(9)
    src = rng.integers(0, 256, size=pool, dtype=np.uint8)
    dst = np.full(pool, 0x5A, dtype=np.uint8)
    oracle.copy_fragments(src, dst, frags)
    covered = np.zeros(pool, dtype=bool)
    for s, d, ln in frags.astype(np.int64):
        assert not covered[d:d + ln].any()          # generator keeps dst disjoint
        covered[d:d + ln] = True
        assert np.array_equal(dst[d:d + ln], src[s:s + ln])
    assert np.all(dst[~covered] == 0x5A)
    assert covered.sum() == frags[:, 2].sum()       # bytes conserved
    # order independence
    dst2 = np.full(pool, 0x5A, dtype=np.uint8)
    oracle.copy_fragments(src, dst2, frags[rng.permutation(n)])
    assert np.array_equal(dst, dst2)


def test_copy_single_fragment_is_plain_copy():
    rng = np.random.default_rng(10)
    src = rng.integers(0, 256, size=1 << 20, dtype=np.uint8)
    dst = np.zeros_like(src)
    oracle.copy_fragments(src, dst, np.array([[0, 0, src.size]], dtype=np.uint64))
    ref = np.empty_like(src)
    np.copyto(ref, src)
    assert np.array_equal(dst, ref)
    oracle.copy_fragments(src, dst, np.zeros((0, 3), dtype=np.uint64))   # empty list
    oracle.copy_fragments(src, dst, np.array([[5, 7, 0]], dtype=np.uint64))  # len 0


def test_moe_permutation_then_inverse_is_identity():
    E, n = 4096, 64
    frags, perm = synth.moe_permutation(n, E, seed=12)
    rng = np.random.default_rng(13)
    src = rng.integers(0, 256, size=n * E, dtype=np.uint8)
    mid = np.zeros_like(src)
    oracle.copy_fragments(src, mid, frags)
    # slot j holds expert perm[j]
    assert np.array_equal(mid.reshape(n, E), src.reshape(n, E)[perm])
    inv = np.stack([np.arange(n) * E, perm * E, np.full(n, E)], axis=1).astype(np.uint64)
    back = np.zeros_like(src)
    oracle.copy_fragments(mid, back, inv)
    assert np.array_equal(back, src)


def test_tp_shards_reassemble_the_full_weights():
    spec = synth.spec_scaled(layers=2, hidden=256, q_heads=4, kv_heads=2, head_dim=64, mlp=384)
    n = synth.spec_elems(spec)
    stream = np.arange(n, dtype=np.int64)           # every element distinct
    tp = 4
    shards = [oracle.tp_shard(stream, spec, tp, r) for r in range(tp)]
    assert sum(s.size for s in shards) == n          # bytes conserved
    assert np.array_equal(oracle.tp_shard(stream, spec, 1, 0), stream)  # tp=1 is identity
    off = [0] * tp
    soff = 0
    for (_, rows, cols, split) in spec:
        w = torch.from_numpy(stream[soff:soff + rows * cols].reshape(rows, cols))
        soff += rows * cols
        dim = 0 if split == "rows" else 1
        ref = torch.chunk(w, tp, dim=dim)
        parts = []
        for r in range(tp):
            k = ref[r].numel()
            got = shards[r][off[r]:off[r] + k].reshape(ref[r].shape)
            off[r] += k
            assert np.array_equal(got, ref[r].contiguous().numpy())
            parts.append(torch.from_numpy(got))
        assert torch.equal(torch.cat(parts, dim=dim), w)


def test_zipf_ids_distinct_and_skewed():
    ids = synth.ids_zipf_prefix_reuse(32768, 4096, 1.1, seed=1002)
    assert ids.dtype == np.int32 and len(ids) == 4096 and len(np.unique(ids)) == 4096
    assert ids.min() >= 0 and ids.max() < 32768
    raw = synth.ids_zipf_prefix_reuse(32768, 4096, 1.1, seed=1002, keep_duplicates=True)
    assert len(np.unique(raw)) < 4096                # prefix reuse repeats blocks


def _fletcher64_recurrence(data: bytes):
    """Sequential Fletcher-style sums: A_k = A_(k-1) + b_k, B_k = B_(k-1) + A_k."""
    a = b = 0
    for x in data:
        a = (a + x) % (1 << 64)
        b = (b + a) % (1 << 64)
    return a, b


def test_digests_hand_values_and_fletcher_relation():
    buf = np.array([1, 2, 3, 250, 0, 7], dtype=np.uint8)
    d = oracle.fragment_digests(buf, np.array([[0, 0, 3], [3, 0, 3], [0, 0, 0]], dtype=np.uint64))
    assert d[0].tolist() == [6, 1 * 1 + 2 * 2 + 3 * 3]
    assert d[1].tolist() == [257, 250 + 0 + 21]
    assert d[2].tolist() == [0, 0]
    # the weighted sum equals (n + 1) * A_n - B_n of the sequential recurrence
    rng = np.random.default_rng(90)
    data = rng.integers(0, 256, size=5000, dtype=np.int64).astype(np.uint8)
    a, b = _fletcher64_recurrence(bytes(data))
    s = oracle.fragment_digests(data, np.array([[0, 0, data.size]], dtype=np.uint64))[0]
    assert int(s[0]) == a == int(data.astype(np.uint64).sum())
    assert int(s[1]) == ((data.size + 1) * a - b) % (1 << 64)


def test_digests_detect_swaps_and_use_dst_offsets():
    rng = np.random.default_rng(91)
    buf = rng.integers(0, 256, size=4096, dtype=np.int64).astype(np.uint8)
    f = np.array([[100, 1000, 777]], dtype=np.uint64)
    d0 = oracle.fragment_digests(buf, f)
    swapped = buf.copy()
    i, j = 150, 400
    assert swapped[i] != swapped[j]
    swapped[i], swapped[j] = swapped[j], swapped[i]
    d1 = oracle.fragment_digests(swapped, f)
    assert d1[0, 0] == d0[0, 0] and d1[0, 1] != d0[0, 1]    # same bytes, different order
    dd = oracle.fragment_digests(np.roll(buf, 900), f, use_src=False)
    assert np.array_equal(dd, d0)                             # dst_off 1000 holds src bytes from 100
