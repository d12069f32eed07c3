"""GPU parity: fragment copies and tensor-parallel shard materialization.

HIP path through the C ABI against the CPU oracle, byte for byte, on the
same seeded inputs: small storms (aligned and byte-granular), edge cases,
planned reuse, MoE expert permutations, a TP=8 shard of 8B-shaped weights,
and the full-size fragment storm.
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


def _host(t):
    return t.detach().to("cpu").numpy()


def _rand_bytes(n, seed):
    return synth.random_bytes(n, seed, device=DEV)


def _copy_and_check(src, frags_np, dst_size, sentinel=0x5A, planned=False, ws_bytes=None):
    frags = torch.from_numpy(frags_np.astype(np.uint64).view(np.int64)).to(DEV)
    dst = torch.full((dst_size,), sentinel, dtype=torch.uint8, device=DEV)
    n = len(frags_np)
    if ws_bytes is None:
        ws_bytes = tc.tc_copy_fragments_workspace(n)
    ws = torch.empty(max(ws_bytes, 8), dtype=torch.uint8, device=DEV)
    if planned:
        total = tc.tc_plan_fragments(frags, ws)
        tc.tc_copy_planned(src, dst, ws, total)
        ws.total = total
    else:
        tc.tc_copy_fragments(src, dst, frags, ws)
    torch.cuda.synchronize()
    want = np.full(dst_size, sentinel, dtype=np.uint8)
    oracle.copy_fragments(_host(src), want, frags_np)
    got = _host(dst)
    step = 1 << 28
    for a in range(0, dst_size, step):
        g, w = got[a:a + step], want[a:a + step]
        if not np.array_equal(g, w):
            bad = np.nonzero(g != w)[0]
            raise AssertionError(f"{bad.size} bytes differ in chunk at {a}, first at {bad[:5] + a}")
    return dst, frags, ws


@pytest.mark.parametrize("align", [16, 4, 1])
def test_storm_small(align):
    pool = 256 << 20
    frags = synth.fragment_storm(20000, pool, seed=31 + align, align=align)
    _copy_and_check(_rand_bytes(pool, 32), frags, pool)


def test_every_residue_pair_and_ragged_length():
    """Every source offset mod 16 against every destination offset mod 128
    (the vector path's and the line cut's residues), each with lengths
    around the vector, piece and line boundaries: 26,624 fragments, copied
    with digests, against the oracle."""
    lens = [0, 1, 15, 16, 17, 127, 128, 129, 1023, 1024, 1025, 2175, 4097]
    rows = []
    so = do = 0
    for rs in range(16):
        for rd in range(128):
            for ln in lens:
                so = (so + 15) // 16 * 16 + rs
                do = (do + 127) // 128 * 128 + rd
                rows.append((so, do, ln))
                so += ln + 5
                do += ln + 7
    frags = np.array(rows, dtype=np.uint64)
    n = len(frags)
    src = _rand_bytes(so + 16, 95)
    dst_size = do + 16
    dst, fr, ws = _copy_and_check(src, frags, dst_size, planned=True)
    dg = torch.empty(2 * n, dtype=torch.int64, device=DEV)
    dst2 = torch.full((dst_size,), 0x5A, dtype=torch.uint8, device=DEV)
    tc.tc_copy_planned_digest(src, dst2, ws, ws.total, n, dg)
    torch.cuda.synchronize()
    assert torch.equal(dst2, dst)
    got = _host(dg).view(np.uint64).reshape(n, 2)
    assert np.array_equal(got, oracle.fragment_digests(_host(src), frags, use_src=True))


def test_mixed_misalignment():
    """src and dst with different residues mod 16 (byte path), and equal
    residues that are not 0 (vector body with byte head/tail)."""
    rng = np.random.default_rng(33)
    rows = []
    off_s = off_d = 0
    for k in range(3000):
        ln = int(rng.integers(0, 40000))
        ps, pd = int(rng.integers(0, 16)), int(rng.integers(0, 16))
        if k % 2:
            pd = ps
        rows.append((off_s + ps, off_d + pd, ln))
        off_s += ps + ln + 16
        off_d += pd + ln + 16
    frags = np.array(rows, dtype=np.uint64)
    _copy_and_check(_rand_bytes(off_s, 34), frags, off_d)


def test_edge_fragments():
    src = _rand_bytes(4 << 20, 35)
    rows = [(0, 0, 0), (5, 9, 0)]                          # empty fragments
    rows += [(100, 200, 1), (1000, 300, 15), (2000, 400, 16), (3000, 500, 17)]
    rows += [(16, 1 << 20, (1 << 20) + 3)]                 # larger than a piece, ragged
    rows += [(3 << 20, 5 << 19, 16384), (7 << 19, 11 << 18, 16385)]
    rows += [(2048 + k, 8192 + 4 * k, 0) for k in range(50)]  # many zero-length in a row
    _copy_and_check(src, np.array(rows, dtype=np.uint64), 4 << 20)
    # single fragment covering the whole buffer = plain copy
    _copy_and_check(src, np.array([(0, 0, 4 << 20)], dtype=np.uint64), 4 << 20)
    # nothing to do
    empty = torch.zeros((0, 3), dtype=torch.int64, device=DEV)
    tc.tc_copy_fragments(src, src, empty, torch.empty(8, dtype=torch.uint8, device=DEV))


def test_plan_reuse_and_order_independence():
    pool = 64 << 20
    frags = synth.fragment_storm(5000, pool, seed=36)
    src = _rand_bytes(pool, 37)
    dst, fr, ws = _copy_and_check(src, frags, pool, planned=True)
    # the same plan again
    dst2 = torch.full_like(dst, 0x5A)
    tc.tc_copy_planned(src, dst2, ws, ws.total)
    # a shuffled list planned afresh gives the same bytes
    perm = np.random.default_rng(38).permutation(len(frags))
    dst3, _, _ = _copy_and_check(src, frags[perm], pool)
    torch.cuda.synchronize()
    assert torch.equal(dst, dst2) and torch.equal(dst, dst3)


@pytest.mark.parametrize("extra_tasks", [1, 100, 5000])
def test_small_workspace_grows_the_task_size(extra_tasks):
    """With room for only n + k tasks the plan picks larger pieces; the copy
    must not change."""
    pool = 64 << 20
    frags = synth.fragment_storm(3000, pool, seed=42)
    n = len(frags)
    ws_bytes = tc.tc_copy_fragments_workspace_min(n) + 32 * (extra_tasks - 1)
    src = _rand_bytes(pool, 43)
    dst, fr, ws = _copy_and_check(src, frags, pool, planned=True, ws_bytes=ws_bytes)
    assert ws.total <= n + extra_tasks + 32      # capacity rounds to 256-byte alignment
    assert _header_word(ws, 8) == 0               # larger pieces: plain multiples
    with pytest.raises(tc.TcError) as e:          # below the minimum
        tc.tc_plan_fragments(fr, torch.empty(tc.tc_copy_fragments_workspace_min(n) - 4096,
                                             dtype=torch.uint8, device=DEV))
    assert e.value.status == 5


def test_validation_mode_reports_overlaps():
    src = _rand_bytes(1 << 20, 39)
    dst = torch.zeros(1 << 20, dtype=torch.uint8, device=DEV)
    ws = torch.empty(tc.tc_copy_fragments_workspace(2), dtype=torch.uint8, device=DEV)
    bad = torch.tensor([[0, 0, 100], [200, 50, 100]], dtype=torch.int64, device=DEV)
    tc.tc_set_validate(True)
    try:
        with pytest.raises(tc.TcError) as e:
            tc.tc_copy_fragments(src, dst, bad, ws)
        assert e.value.status == 3
        same = torch.tensor([[0, 50, 100]], dtype=torch.int64, device=DEV)
        with pytest.raises(tc.TcError) as e:       # src and dst ranges overlap in one buffer
            tc.tc_copy_fragments(src, src, same, ws)
        assert e.value.status == 3
        huge = torch.tensor([[0, (1 << 48) - 8, 100]], dtype=torch.int64, device=DEV)
        with pytest.raises(tc.TcError) as e:       # offsets must stay below 2^48
            tc.tc_copy_fragments(src, dst, huge, ws)
        assert e.value.status == 2
    finally:
        tc.tc_set_validate(False)


def test_moe_permutation_small_and_full():
    for n_exp, e_bytes in [(32, 65536), (256, 7168 * 2048)]:
        frags, perm = synth.moe_permutation(n_exp, e_bytes, seed=synth.SEED_STORM)
        src = _rand_bytes(n_exp * e_bytes, 40)
        fr = torch.from_numpy(frags.view(np.int64)).to(DEV)
        dst = torch.empty_like(src)
        ws = torch.empty(tc.tc_copy_fragments_workspace(n_exp), dtype=torch.uint8, device=DEV)
        tc.tc_copy_fragments(src, dst, fr, ws)
        torch.cuda.synchronize()
        # expert slot j holds source expert perm[j] (torch indexing on the device)
        p = torch.from_numpy(perm).to(DEV)
        assert torch.equal(dst.view(n_exp, e_bytes), src.view(n_exp, e_bytes)[p])
        # every expert against the oracle's copy of the same descriptors
        want = np.zeros(n_exp * e_bytes, dtype=np.uint8)
        oracle.copy_fragments(_host(src), want, frags)
        assert np.array_equal(_host(dst), want)
        del src, dst, want


@pytest.mark.parametrize("layers,tp,ranks", [(2, 8, range(8)), (32, 8, [3])])
def test_tp_shard_8b(layers, tp, ranks):
    """8B-shaped weights (q/o 4096x4096, k/v 1024x4096, gate/up 14336x4096,
    down 4096x14336) in a contiguous bf16 stream, materialized into TP=8
    shards through the builder's fragments and the fragment copy."""
    spec = synth.spec_8b(layers)
    n = synth.spec_elems(spec)
    stream = synth.bf16_normal(n, 1.0, synth.SEED_RESHARD_8B, device=DEV)
    v = tcv.stream_views(spec, tp)
    shard_n = tcv.shard_elems(spec, tp)
    for rank in ranks:
        frags_np = tc.tc_tp_fragments(v, tp, rank)
        frags = torch.from_numpy(frags_np.view(np.int64)).to(DEV)
        ws = torch.empty(tc.tc_copy_fragments_workspace(len(frags_np)), dtype=torch.uint8, device=DEV)
        shard = torch.empty(shard_n, dtype=torch.bfloat16, device=DEV)
        tc.tc_copy_fragments(stream, shard, frags, ws)
        torch.cuda.synchronize()
        got = _host(shard.view(torch.int16)).view(np.uint16)
        if layers <= 2:
            want = oracle.tp_shard(_host(stream.view(torch.int16)).view(np.uint16), spec, tp, rank)
            assert np.array_equal(got, want)
        else:
            # full size: per layer, the oracle's slices of that layer's weights
            per_layer = synth.spec_elems(spec[:7])
            shard_layer = tcv.shard_elems(spec[:7], tp)
            for l in [0, 1, 17, layers - 1]:
                lw = _host(stream[l * per_layer:(l + 1) * per_layer].view(torch.int16)).view(np.uint16)
                want = oracle.tp_shard(lw, spec[7 * l:7 * l + 7], tp, rank)
                assert np.array_equal(got[l * shard_layer:(l + 1) * shard_layer], want)
            # every layer: torch slicing on the device
            off_s = off_d = 0
            for (_, rows, cols, split) in spec:
                w = stream[off_s:off_s + rows * cols].view(rows, cols)
                off_s += rows * cols
                sl = w[rank * rows // tp:(rank + 1) * rows // tp] if split == "rows" else \
                    w[:, rank * cols // tp:(rank + 1) * cols // tp]
                k = sl.numel()
                assert torch.equal(shard[off_d:off_d + k].view(sl.shape).view(torch.int16),
                                   sl.contiguous().view(torch.int16))
                off_d += k
    del stream
    torch.cuda.empty_cache()


def test_storm_full_size():
    """1,000,000 fragments, log-uniform 64 B - 64 KiB, in two 16 GiB pools,
    compared in full with the oracle run on host copies."""
    pool = 16 << 30
    frags = synth.fragment_storm(1_000_000, pool, seed=synth.SEED_STORM)
    src = _rand_bytes(pool, synth.SEED_STORM)
    dst, _, _ = _copy_and_check(src, frags, pool)
    del src, dst
    torch.cuda.empty_cache()


def _torch_shards(stream, spec, tp):
    """All tp shards of a contiguous stream, rank-major, built with torch
    slicing on the device (independent of the library)."""
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


@pytest.mark.parametrize("src_tp,dst_tp,ranks", [(8, 4, range(4)), (4, 8, [0, 3, 7]), (8, 1, [0]),
                                                 (2, 8, [5])])
def test_cross_layout_reshard_8b(src_tp, dst_tp, ranks):
    """2 layers of the 8B shapes stored as src_tp shards, rearranged into
    dst_tp shards by the builder's fragments and the planned copy."""
    spec = synth.spec_8b(2)
    n = synth.spec_elems(spec)
    stream = synth.bf16_normal(n, 1.0, synth.SEED_RESHARD_8B, device=DEV)
    src = _torch_shards(stream, spec, src_tp)
    host = _host(stream.view(torch.int16)).view(np.uint16)
    views = tcv.reshard_views(spec, src_tp, dst_tp)
    for rank in ranks:
        frags_np = tc.tc_reshard_fragments(views, dst_tp, rank)
        frags = torch.from_numpy(frags_np.view(np.int64)).to(DEV)
        ws = torch.empty(tc.tc_copy_fragments_workspace(len(frags_np)), dtype=torch.uint8, device=DEV)
        total = tc.tc_plan_fragments(frags, ws)
        dst = torch.empty(tcv.shard_elems(spec, dst_tp), dtype=torch.bfloat16, device=DEV)
        tc.tc_copy_planned(src, dst, ws, total)
        torch.cuda.synchronize()
        want = oracle.tp_shard(host, spec, dst_tp, rank)
        assert np.array_equal(_host(dst.view(torch.int16)).view(np.uint16), want)


def test_cross_layout_reshard_8b_full_size():
    """32 layers of the 8B shapes: the TP=8 shards (13.96 GB) rearranged into
    TP=4 rank 1; every slice checked against torch slicing of the stream on
    the device, two layers against the oracle."""
    spec = synth.spec_8b(32)
    n = synth.spec_elems(spec)
    stream = synth.bf16_normal(n, 1.0, synth.SEED_RESHARD_8B, device=DEV)
    src = _torch_shards(stream, spec, 8)
    frags_np = tc.tc_reshard_fragments(tcv.reshard_views(spec, 8, 4), 4, 1)
    frags = torch.from_numpy(frags_np.view(np.int64)).to(DEV)
    ws = torch.empty(tc.tc_copy_fragments_workspace(len(frags_np)), dtype=torch.uint8, device=DEV)
    total = tc.tc_plan_fragments(frags, ws)
    dst = torch.empty(tcv.shard_elems(spec, 4), dtype=torch.bfloat16, device=DEV)
    tc.tc_copy_planned(src, dst, ws, total)
    torch.cuda.synchronize()
    want = _torch_shards(stream, spec, 4)[1 * dst.numel():2 * dst.numel()]
    assert torch.equal(dst.view(torch.int16), want.view(torch.int16))
    per_layer = synth.spec_elems(spec[:7])
    shard_layer = tcv.shard_elems(spec[:7], 4)
    got = _host(dst.view(torch.int16)).view(np.uint16)
    for l in [0, 31]:
        lw = _host(stream[l * per_layer:(l + 1) * per_layer].view(torch.int16)).view(np.uint16)
        assert np.array_equal(got[l * shard_layer:(l + 1) * shard_layer],
                              oracle.tp_shard(lw, spec[7 * l:7 * l + 7], 4, 1))


def _header_permuted(ws):
    # the plan header's eighth word says whether the tasks follow a reordered list
    return int(ws[56:64].cpu().numpy().view(np.uint64)[0])


def _header_word(ws, k):
    return int(ws[8 * k:8 * k + 8].cpu().numpy().view(np.uint64)[0])


def _task_table(ws):
    t = ws[256:256 + 16 * ws.total].cpu().numpy().view(np.uint64).reshape(-1, 2)
    src = t[:, 0] & np.uint64((1 << 48) - 1)
    dst = (t[:, 0] >> np.uint64(48)) | ((t[:, 1] & np.uint64(0xFFFFFFFF)) << np.uint64(16))
    ln = (t[:, 1] >> np.uint64(32)) & np.uint64(0x7FFFFFFF)
    first = (t[:, 1] >> np.uint64(63)).astype(bool)
    return src.astype(np.int64), dst.astype(np.int64), ln.astype(np.int64), first


@pytest.mark.parametrize("align", [16, 1])
def test_tasks_start_on_destination_lines(align):
    """1 KiB pieces are cut on 128-byte destination lines: every task after a
    fragment's first starts at a multiple of 128 in the destination, the
    first is the shorter by the fragment's offset into its line, and the
    tasks of each fragment tile it exactly (checked from the task table)."""
    pool = 64 << 20
    frags = synth.fragment_storm(3000, pool, seed=47 + align, align=align)
    _, _, ws = _copy_and_check(_rand_bytes(pool, 48), frags, pool, planned=True)
    assert _header_word(ws, 1) == 1024 and _header_word(ws, 8) == 127
    src, dst, ln, first = _task_table(ws)
    assert np.all(dst[~first] % 128 == 0)
    assert first.sum() == np.count_nonzero(frags[:, 2])
    assert np.all(ln > 0) and np.all(ln <= 1024)
    # each fragment's tasks, in plan order, tile its bytes
    fid = np.cumsum(first) - 1
    nz = np.nonzero(frags[:, 2])[0]
    f = frags[nz].astype(np.int64)[fid]
    off = dst - f[:, 1]
    assert np.array_equal(src - f[:, 0], off)
    nxt = np.append(off[1:], 0)
    last = np.append(first[1:], True)
    assert np.array_equal(np.where(last, f[:, 2], nxt), off + ln)
    h = f[:, 1] % 128
    assert np.array_equal(ln[first], np.minimum(f[first, 2], 1024 - h[first]))


def test_long_unordered_lists_are_planned_in_destination_order():
    """A list of 5,000 fragments with scattered destinations is planned in
    destination order; an ordered list, and an unordered one of 1,000, keep
    their order.  The copies are exact either way."""
    pool = 64 << 20
    src = _rand_bytes(pool, 44)
    frags = synth.fragment_storm(5000, pool, seed=45)
    _, _, ws = _copy_and_check(src, frags, pool, planned=True)
    assert _header_permuted(ws) == 1
    # the task table ascends in destination address at bucket granularity
    # (64 KiB buckets here): consecutive tasks never step back by 1 MiB or more,
    # while the list as given does
    tasks = ws[256:256 + 16 * ws.total].cpu().numpy().view(np.uint64).reshape(-1, 2)
    dst = (tasks[:, 0] >> np.uint64(48)) | ((tasks[:, 1] & np.uint64(0xFFFFFFFF)) << np.uint64(16))
    assert np.diff(dst.astype(np.int64)).min() > -(1 << 20)
    assert np.diff(frags[:, 1].astype(np.int64)).min() < -(1 << 20)
    ordered = frags[np.argsort(frags[:, 1], kind="stable")]
    _, _, ws2 = _copy_and_check(src, ordered, pool, planned=True)
    assert _header_permuted(ws2) == 0
    _, _, ws3 = _copy_and_check(src, synth.fragment_storm(1000, pool, seed=46), pool, planned=True)
    assert _header_permuted(ws3) == 0


def test_fragment_longer_than_4gib_beyond_4gib():
    """One fragment of 4 GiB + 17 bytes, read from and written to offsets past
    2^32, beside two small ones: 64-bit offsets and lengths in the plan, the
    copy and the digests.  The copy checked in full on the device and, in
    sampled windows, against the oracle; the digests against the oracle."""
    big = (4 << 30) + 17
    src_size, dst_size = (5 << 30) + 4096, (6 << 30) + 4096
    src = _rand_bytes(src_size, 47)
    rows = np.array([((1 << 30) + 3, (3 << 30) // 2 + 3, big),   # same residue: vector body
                     (100, 200, 1000), (5 << 30, 8192, 4096)], dtype=np.uint64)
    frags = torch.from_numpy(rows.view(np.int64)).to(DEV)
    dst = torch.full((dst_size,), 0x5A, dtype=torch.uint8, device=DEV)
    ws = torch.empty(tc.tc_copy_fragments_workspace(3), dtype=torch.uint8, device=DEV)
    tc.tc_copy_fragments(src, dst, frags, ws)
    torch.cuda.synchronize()
    s0, d0 = int(rows[0, 0]), int(rows[0, 1])
    assert torch.equal(dst[d0:d0 + big], src[s0:s0 + big])
    assert torch.equal(dst[200:1200], src[100:1100]) and torch.equal(dst[8192:12288], src[5 << 30:(5 << 30) + 4096])
    for a, b in ((0, 200), (1200, 8192), (12288, d0), (d0 + big, dst_size)):
        assert int((dst[a:b] != 0x5A).sum()) == 0, (a, b)
    for off in (0, (1 << 32) - 8192, big - 4096):
        w = np.zeros(4096, np.uint8)
        oracle.copy_fragments(_host(src[s0 + off:s0 + off + 4096]), w, np.array([[0, 0, 4096]], np.uint64))
        assert np.array_equal(_host(dst[d0 + off:d0 + off + 4096]), w)
    # digests over the same fragments: byte positions past 2^32 in a fragment
    # and destination offsets past 2^32 in the weights
    total = tc.tc_plan_fragments(frags, ws)
    dg = torch.empty(6, dtype=torch.int64, device=DEV)
    dd = torch.empty(6, dtype=torch.int64, device=DEV)
    tc.tc_digest_planned(src, tc.DIGEST_SRC, ws, total, 3, dg)
    tc.tc_digest_planned(dst, tc.DIGEST_DST, ws, total, 3, dd)
    torch.cuda.synchronize()
    want = oracle.fragment_digests(_host(src), rows, use_src=True)
    assert np.array_equal(_host(dg).view(np.uint64).reshape(3, 2), want)
    assert np.array_equal(_host(dd).view(np.uint64).reshape(3, 2), want)
    del src, dst
    torch.cuda.empty_cache()


def test_plan_of_more_than_16m_fragments():
    """A list longer than 16,384 count blocks (17M fragments of 64 bytes,
    destinations unordered): the plan takes the block prefix from its own
    offsets pass and reorders the list; the asynchronous one-call copy, a
    planned copy and the plan's task count against the oracle."""
    n = 17_000_000
    pool = 2 << 30
    print(f"case: {n} fragments of 64 B in 2 GiB pools", flush=True)
    frags = synth.fragment_storm(n, pool, seed=77, lo=64, hi=64)
    src = _rand_bytes(pool, 78)
    fr = torch.from_numpy(frags.view(np.int64)).to(DEV)
    ws = torch.empty(tc.tc_copy_fragments_workspace(n), dtype=torch.uint8, device=DEV)
    dst = torch.full((pool,), 0x5A, dtype=torch.uint8, device=DEV)
    tc.tc_copy_fragments(src, dst, fr, ws)
    total = tc.tc_plan_status(ws)
    assert total == n                                  # 64 B plus a line offset fit one piece
    assert _header_word(ws, 7) == 1                    # reordered
    dst2 = torch.full_like(dst, 0x5A)
    tc.tc_copy_planned(src, dst2, ws, total)
    torch.cuda.synchronize()
    want = np.full(pool, 0x5A, dtype=np.uint8)
    oracle.copy_fragments(_host(src), want, frags)
    assert np.array_equal(_host(dst), want)
    assert np.array_equal(_host(dst2), want)
