"""GPU parity: fragment copies with integrity digests.

The copy-with-digest and digest-only entry points against the oracle's
per-fragment digests and its copy, on the same seeded inputs: storms
(aligned and byte-granular), empty fragments, fragments laid back to back,
fragments spanning many reduction windows, long runs of empty descriptors, plans with pieces larger
than 1 KiB, and the full-size cross-layout shard copy.
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


def _plan(frags_np, ws_bytes=None):
    frags = torch.from_numpy(np.ascontiguousarray(frags_np, dtype=np.uint64).view(np.int64)).to(DEV)
    n = len(frags_np)
    if ws_bytes is None:
        ws_bytes = tc.tc_copy_fragments_workspace(n)
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=DEV)
    total = tc.tc_plan_fragments(frags, ws)
    return frags, ws, total


def _digests(n):
    # garbage first: every word must be written
    return torch.full((max(2 * n, 1),), -1, dtype=torch.int64, device=DEV)


def _as_u64(t, n):
    return _host(t)[:2 * n].view(np.uint64).reshape(n, 2)


def _check(src, frags_np, dst_size, ws_bytes=None, sentinel=0x3C):
    n = len(frags_np)
    frags, ws, total = _plan(frags_np, ws_bytes)
    dst = torch.full((dst_size,), sentinel, dtype=torch.uint8, device=DEV)
    dg, ds, dd = _digests(n), _digests(n), _digests(n)
    tc.tc_copy_planned_digest(src, dst, ws, total, n, dg)
    tc.tc_digest_planned(src, tc.DIGEST_SRC, ws, total, n, ds)
    tc.tc_digest_planned(dst, tc.DIGEST_DST, ws, total, n, dd)
    torch.cuda.synchronize()
    hsrc = _host(src)
    want = oracle.fragment_digests(hsrc, frags_np, use_src=True)
    got = _as_u64(dg, n)
    bad = np.nonzero(np.any(got != want, axis=1))[0]
    assert bad.size == 0, f"{bad.size} digests differ, first fragments {bad[:5]}"
    assert np.array_equal(_as_u64(ds, n), want)
    assert np.array_equal(_as_u64(dd, n), want)
    ref = np.full(dst_size, sentinel, dtype=np.uint8)
    oracle.copy_fragments(hsrc, ref, frags_np)
    assert np.array_equal(_host(dst), ref)
    return total, ws


@pytest.mark.parametrize("align", [16, 1])
def test_digest_storm_small(align):
    pool = 64 << 20
    frags = synth.fragment_storm(5000, pool, seed=71 + align, align=align)
    _check(synth.random_bytes(pool, 72, device=DEV), frags, pool)


def test_digest_edges_and_misalignment():
    src = synth.random_bytes(8 << 20, 73, device=DEV)
    rows = [(0, 0, 0), (5, 9, 0)]
    rows += [(100, 200, 1), (1001, 300, 15), (2000, 400, 16), (3003, 503, 17), (4100, 4200, 1025)]
    rows += [(16, 1 << 20, (1 << 20) + 3)]                    # many pieces, ragged end
    rows += [(3 << 20, 5 << 19, 16384), (7 << 19, 11 << 18, 16385)]
    rows += [(2048 + k, 8192 + 4 * k, 0) for k in range(50)]  # zero-length run
    rows += [(5 << 20 | 5, 6 << 20 | 5, 4097)]                  # equal residues, not 0
    rows += [(6 << 20 | 3, 7 << 20 | 9, 3000)]                  # different residues: byte path
    _check(src, np.array(rows, dtype=np.uint64), 8 << 20)


def test_digest_fragment_spanning_many_windows():
    """A 96 MiB fragment (98,304 tasks of 1 KiB, 96 reduction windows) between
    two small ones: its digest is summed across windows atomically."""
    src = synth.random_bytes(100 << 20, 74, device=DEV)
    rows = np.array([(0, 0, 777), (4096, 4096, 96 << 20), ((97 << 20), (97 << 20), 5000)],
                    dtype=np.uint64)
    total, _ = _check(src, rows, 100 << 20)
    assert total > 96 * 1024


def test_digest_long_runs_of_empty_descriptors():
    """2,000 empty descriptors between two 512-task fragments put both in one
    window whose fragment span exceeds the window (the global-search path)."""
    src = synth.random_bytes(4 << 20, 75, device=DEV)
    rows = [(0, 0, 512 << 10)]
    rows += [(123, 456, 0)] * 2000
    rows += [(1 << 20, 1 << 20, 512 << 10)]
    rows += [(7, 7, 0)] * 3000
    rows += [(2 << 20, 2 << 20, 700 << 10), (3 << 20, 3 << 20, 3)]
    _check(src, np.array(rows, dtype=np.uint64), 4 << 20)


def _back_to_back(n, seed, reverse_dst):
    """n fragments of 1-8 KiB, some ragged, laid end to end in the source and
    in the destination (in reverse order when reverse_dst), so consecutive
    tasks of different fragments are contiguous on the side being summed."""
    rng = np.random.default_rng(seed)
    lens = 1024 * rng.integers(1, 9, size=n) + rng.choice([0, 0, 0, 16, 5, 1000 - 1024], size=n)
    src = np.concatenate([[0], np.cumsum(lens)[:-1]])
    order = np.arange(n)[::-1] if reverse_dst else np.arange(n)
    dst = np.empty(n, dtype=np.int64)
    dst[order] = np.concatenate([[0], np.cumsum(lens[order])[:-1]])
    return np.stack([src, dst, lens], axis=1).astype(np.uint64), int(lens.sum())


@pytest.mark.parametrize("n,reverse_dst", [(2000, False), (5000, True)])
def test_digest_adjacent_fragments_stay_separate(n, reverse_dst):
    """Tasks summed as one run must belong to one fragment: with fragments
    back to back, a group of consecutive tasks crossing a fragment boundary
    covers contiguous bytes, and only the fragment boundary keeps the two
    digests apart.  5000 fragments with descending destinations take the
    destination-ordered plan."""
    frags, payload = _back_to_back(n, 81 + n, reverse_dst)
    _check(synth.random_bytes(payload, 82, device=DEV), frags, payload)


@pytest.mark.parametrize("extra_tasks", [1, 300])
def test_digest_with_pieces_larger_than_1k(extra_tasks):
    pool = 64 << 20
    frags = synth.fragment_storm(3000, pool, seed=76)
    n = len(frags)
    ws_bytes = tc.tc_copy_fragments_workspace_min(n) + 32 * (extra_tasks - 1)
    total, ws = _check(synth.random_bytes(pool, 77, device=DEV), frags, pool, ws_bytes=ws_bytes)
    assert total <= n + extra_tasks + 32


def test_digest_all_empty_and_errors():
    src = synth.random_bytes(1 << 16, 78, device=DEV)
    rows = np.array([(0, 0, 0)] * 5, dtype=np.uint64)
    frags, ws, total = _plan(rows)
    assert total == 0
    dg = _digests(5)
    tc.tc_copy_planned_digest(src, src, ws, total, 5, dg)
    torch.cuda.synchronize()
    assert np.all(_as_u64(dg, 5) == 0)
    with pytest.raises(ValueError):               # digest array too small
        tc.tc_copy_planned_digest(src, src, ws, total, 5, _digests(4))
    with pytest.raises(tc.TcError) as e:           # unknown side
        tc.tc_digest_planned(src, 7, ws, total, 5, dg)
    assert e.value.status == 1
    # validation: n must be the plan's descriptor count
    frags_np = synth.fragment_storm(100, 4 << 20, seed=79)
    fr, ws2, total2 = _plan(frags_np)
    src = synth.random_bytes(4 << 20, 80, device=DEV)
    dst = torch.zeros(4 << 20, dtype=torch.uint8, device=DEV)
    tc.tc_set_validate(True)
    try:
        with pytest.raises(tc.TcError) as e:
            tc.tc_copy_planned_digest(src, dst, ws2, total2, 99, _digests(100))
        assert e.value.status == 1
        tc.tc_copy_planned_digest(src, dst, ws2, total2, 100, _digests(100))
    finally:
        tc.tc_set_validate(False)


def _torch_shards(stream, spec, tp):
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


def test_digest_reshard_8b_full_size():
    """The TP=8 shards of 32 layers of 8B-shaped weights rearranged into TP=4
    rank 2 with digests: every digest against the oracle over the host copy of
    the source shards, the copied bytes against torch slicing on the device."""
    spec = synth.spec_8b(32)
    stream = synth.bf16_normal(synth.spec_elems(spec), 1.0, synth.SEED_RESHARD_8B, device=DEV)
    src = _torch_shards(stream, spec, 8)
    want_dst = _torch_shards(stream, spec, 4)
    del stream
    frags_np = tc.tc_reshard_fragments(tcv.reshard_views(spec, 8, 4), 4, 2)
    n = len(frags_np)
    frags, ws, total = _plan(frags_np)
    dst = torch.empty(tcv.shard_elems(spec, 4), dtype=torch.bfloat16, device=DEV)
    dg = _digests(n)
    tc.tc_copy_planned_digest(src, dst, ws, total, n, dg)
    torch.cuda.synchronize()
    k = dst.numel()
    assert torch.equal(dst.view(torch.int16), want_dst[2 * k:3 * k].view(torch.int16))
    del want_dst
    hsrc = _host(src.view(torch.uint8))
    assert np.array_equal(_as_u64(dg, n), oracle.fragment_digests(hsrc, frags_np, use_src=True))


def test_digest_storm_full_size():
    """The timed storm with digests: 1,000,000 fragments in two 16 GiB pools,
    planned in destination order with the line cut; every digest of the
    copy and of a read of the destination against the oracle over the host
    copy of the source."""
    pool = 16 << 30
    frags_np = synth.fragment_storm(1_000_000, pool, seed=synth.SEED_STORM)
    n = len(frags_np)
    src = synth.random_bytes(pool, synth.SEED_STORM, device=DEV)
    frags, ws, total = _plan(frags_np)
    dst = torch.empty(pool, dtype=torch.uint8, device=DEV)
    dg, dd = _digests(n), _digests(n)
    tc.tc_copy_planned_digest(src, dst, ws, total, n, dg)
    tc.tc_digest_planned(dst, tc.DIGEST_DST, ws, total, n, dd)
    torch.cuda.synchronize()
    del dst
    want = oracle.fragment_digests(_host(src), frags_np, use_src=True)
    got = _as_u64(dg, n)
    bad = np.nonzero(np.any(got != want, axis=1))[0]
    assert bad.size == 0, f"{bad.size} digests differ, first fragments {bad[:5]}"
    assert np.array_equal(_as_u64(dd, n), want)
    del src
    torch.cuda.empty_cache()
