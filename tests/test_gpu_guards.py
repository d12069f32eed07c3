"""GPU: guard bands around every output.

Each output buffer is a slice in the middle of a larger allocation whose
bytes before and after it hold a canary; after the call the canaries must be
untouched and the output must equal the oracle's.  Sizes are ragged so that
tails, edge tiles and byte paths run right up to the slice's ends.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_06007_amd as tc

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
GUARD = 4096
CANARY = 0xCD


def _guarded(nbytes, fill=CANARY):
    """(whole allocation, the output slice in its middle)."""
    whole = torch.full((GUARD + nbytes + GUARD,), fill, dtype=torch.uint8, device=DEV)
    return whole, whole[GUARD:GUARD + nbytes]


def _guards_intact(whole, nbytes):
    h = whole.cpu().numpy()
    assert np.all(h[:GUARD] == CANARY), "bytes before the output changed"
    assert np.all(h[GUARD + nbytes:] == CANARY), "bytes after the output changed"


@pytest.mark.parametrize("B,stride", [(8192 + 16, 8192 + 48), (100, 104)])
def test_gather_scatter_guards(B, stride):
    R, nb = 3, 40
    rng = np.random.default_rng(90)
    ids_np = synth.ids_without_replacement(nb, 17, seed=91)
    ids = torch.from_numpy(ids_np).to(DEV)
    region_bytes = (nb - 1) * stride + B
    host = [rng.integers(0, 256, size=region_bytes, dtype=np.uint8) for _ in range(R)]
    src = [torch.from_numpy(h).to(DEV) for h in host]
    out_bytes = len(ids_np) * R * B
    whole, out = _guarded(out_bytes)
    tc.tc_gather_blocks(src, nb, B, stride, ids, out)
    # scatter into regions that are guarded slices of their own allocations
    dst = [_guarded(region_bytes, fill=0x11) for _ in range(R)]
    for w, _ in dst:
        w[:GUARD] = CANARY
        w[GUARD + region_bytes:] = CANARY
    tc.tc_scatter_blocks([r for _, r in dst], nb, B, stride, ids, out)
    torch.cuda.synchronize()
    want = oracle.gather_blocks(host, B, stride, ids_np)
    assert np.array_equal(out.cpu().numpy(), want.reshape(-1))
    _guards_intact(whole, out_bytes)
    hd = [np.full(region_bytes, 0x11, np.uint8) for _ in range(R)]
    oracle.scatter_blocks(hd, B, stride, ids_np, want.reshape(-1))
    for (w, r), h in zip(dst, hd):
        assert np.array_equal(r.cpu().numpy(), h)
        _guards_intact(w, region_bytes)


@pytest.mark.parametrize("align", [16, 1])
def test_fragment_copy_and_digest_guards(align):
    """The last fragment ends exactly at the end of the destination; the
    digest array is guarded too."""
    pool = 32 << 20
    frags = synth.fragment_storm(2000, pool, seed=92 + align, align=align)
    end = int((frags[:, 1] + frags[:, 2]).max())
    src = synth.random_bytes(pool, 93, device=DEV)
    whole, dst = _guarded(end, fill=0x22)
    whole[:GUARD] = CANARY
    whole[GUARD + end:] = CANARY
    n = len(frags)
    fr = torch.from_numpy(frags.view(np.int64)).to(DEV)
    ws = torch.empty(tc.tc_copy_fragments_workspace(n), dtype=torch.uint8, device=DEV)
    total = tc.tc_plan_fragments(fr, ws)
    dg_whole, dg_bytes = _guarded(16 * n)
    dg = dg_bytes.view(torch.int64)
    tc.tc_copy_planned_digest(src, dst, ws, total, n, dg)
    torch.cuda.synchronize()
    hsrc = src.cpu().numpy()
    want = np.full(end, 0x22, np.uint8)
    oracle.copy_fragments(hsrc, want, frags)
    assert np.array_equal(dst.cpu().numpy(), want)
    _guards_intact(whole, end)
    got = dg.cpu().numpy().view(np.uint64).reshape(n, 2)
    assert np.array_equal(got, oracle.fragment_digests(hsrc, frags, use_src=True))
    _guards_intact(dg_whole, 16 * n)


def test_cast_and_dequant_guards():
    """Ragged matrices (edge tiles on both sides), codes, scales and the
    inverse's bf16 output each in a guarded slice."""
    mats = [(0, 300, 257), (300 * 257 + 5, 128, 384), (300 * 257 + 5 + 128 * 384, 1, 129)]
    n_src = mats[-1][0] + 129
    bits = synth.bf16_normal(n_src, 0.02, 94)
    items = np.zeros(len(mats), dtype=tc.CAST_ITEM_DTYPE)
    ditems = np.zeros(len(mats), dtype=tc.DEQUANT_ITEM_DTYPE)
    q_off = s_off = 0
    for k, (so, rows, cols) in enumerate(mats):
        tcn = (cols + 127) // 128
        items[k] = (so, rows, cols, cols, q_off, cols, s_off, tcn)
        ditems[k] = (q_off, rows, cols, cols, q_off, cols, s_off, tcn)
        q_off += rows * cols
        s_off += ((rows + 127) // 128) * tcn
    src = bits.to(DEV)
    qw, q = _guarded(q_off)
    sw, sb = _guarded(4 * s_off)
    ws = torch.empty(tc.tc_cast_fp8_workspace(len(mats)), dtype=torch.uint8, device=DEV)
    tc.tc_cast_fp8_blockscaled(src, q, sb.view(torch.float32), items, ws)
    yw, yb = _guarded(2 * q_off)
    dws = torch.empty(tc.tc_dequant_fp8_workspace(len(mats)), dtype=torch.uint8, device=DEV)
    tc.tc_dequant_fp8_blockscaled(q, sb.view(torch.float32), yb.view(torch.bfloat16), ditems, dws)
    # the elementwise cast at an odd length
    qsw, qs = _guarded(1001)
    tc.tc_cast_fp8_scaled(src[:1001], 0.01, qs)
    torch.cuda.synchronize()
    for whole, nbytes in ((qw, q_off), (sw, 4 * s_off), (yw, 2 * q_off), (qsw, 1001)):
        _guards_intact(whole, nbytes)
    hx = bits.view(torch.int16).numpy().view(np.uint16)
    hq, hs = q.cpu().numpy(), sb.cpu().numpy().view(np.float32)
    hy = yb.cpu().numpy().view(np.uint16)
    for k, (so, rows, cols) in enumerate(mats):
        wq, wsc = oracle.cast_fp8_blockscaled(hx[so:so + rows * cols].reshape(rows, cols))
        o, s0 = int(items[k]["dst_off"]), int(items[k]["scale_off"])
        assert np.array_equal(hq[o:o + rows * cols].reshape(rows, cols), wq)
        assert np.array_equal(hs[s0:s0 + wsc.size].view(np.uint32), wsc.reshape(-1).view(np.uint32))
        assert np.array_equal(hy[o:o + rows * cols].reshape(rows, cols), oracle.dequant_fp8_blockscaled(wq, wsc))
    assert np.array_equal(qs.cpu().numpy(), oracle.cast_fp8_scaled(hx[:1001], 0.01))


@pytest.mark.parametrize("side", ["src", "dst"])
def test_plan_refuses_offsets_past_48_bits(side):
    """A task holds 48-bit offsets, so a non-empty fragment ending past 2^48
    is refused by the plan's count pass on the device, with validation off,
    and nothing is copied: tc_plan_fragments returns the error, and the
    asynchronous tc_copy_fragments copies nothing and leaves the error in the
    plan, where tc_plan_status reads it.  A fragment ending exactly at 2^48
    is planned (the plan only reads descriptors; it is not copied here)."""
    assert not tc.tc_get_validate()
    lim = 1 << 48
    ok = np.array([[0, 0, 4096], [8192, 4096, 100]], dtype=np.uint64)
    bad = ok.copy()
    col = 0 if side == "src" else 1
    bad[1, col] = lim - 50                     # ends 50 bytes past 2^48
    edge = ok.copy()
    edge[1, col] = lim - 100                   # ends exactly at 2^48
    src = synth.random_bytes(1 << 16, 95, device=DEV)
    whole, dst = _guarded(1 << 16, fill=0x33)
    whole[:GUARD] = CANARY
    whole[GUARD + (1 << 16):] = CANARY
    ws = torch.empty(tc.tc_copy_fragments_workspace(2), dtype=torch.uint8, device=DEV)
    fr = torch.from_numpy(bad.view(np.int64)).to(DEV)
    with pytest.raises(tc.TcError) as e:
        tc.tc_plan_fragments(fr, ws)
    assert e.value.status == 2
    tc.tc_copy_fragments(src, dst, fr, ws)       # enqueued; the plan fails on the device
    with pytest.raises(tc.TcError) as e:
        tc.tc_plan_status(ws)
    assert e.value.status == 2
    tc.tc_copy_planned(src, dst, ws, None)        # a failed plan copies nothing
    torch.cuda.synchronize()
    assert bool((dst == 0x33).all())
    _guards_intact(whole, 1 << 16)
    # a fragment longer than 2^48 on its own is refused the same way
    huge = ok.copy()
    huge[1] = (0, 8192, lim + 16)
    with pytest.raises(tc.TcError) as e:
        tc.tc_plan_fragments(torch.from_numpy(huge.view(np.int64)).to(DEV), ws)
    assert e.value.status == 2
    assert tc.tc_plan_fragments(torch.from_numpy(edge.view(np.int64)).to(DEV), ws) > 0
    torch.cuda.synchronize()
