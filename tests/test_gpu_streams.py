"""GPU: stream ordering and HIP-graph capture of the entry points.

Each call runs on a side stream right behind a device fill that produces its
input on that same stream, so a call that ignored its stream argument would
read stale bytes.  Every call that only enqueues kernels (block
gather/scatter, the asynchronous plan, the one-call fragment copy, planned
copies with and without digests, the block-scaled cast and its inverse in
their one-call and planned forms, the scaled cast) is also captured into a
HIP graph and replayed several times, with the input changed eagerly between
replays and the host item tables overwritten after the capture; every replay
is checked against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_06007_amd as tc

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _pool(R, nb, B):
    flat = torch.zeros(R * nb * B, dtype=torch.uint8, device=DEV)
    return flat, [flat[r * nb * B:(r + 1) * nb * B] for r in range(R)]


def test_side_stream_ordering():
    R, nb, B = 8, 512, 16384
    ids_np = synth.ids_without_replacement(nb, 300, seed=61)
    ids = torch.from_numpy(ids_np).to(DEV)
    src_flat, src = _pool(R, nb, B)
    dst_flat, dst = _pool(R, nb, B)
    buf = torch.empty(300 * R * B, dtype=torch.uint8, device=DEV)
    frags_np = synth.fragment_storm(3000, 32 << 20, seed=62)
    frags = torch.from_numpy(frags_np.view(np.int64)).to(DEV)
    fsrc = torch.empty(32 << 20, dtype=torch.uint8, device=DEV)
    fdst = torch.zeros(32 << 20, dtype=torch.uint8, device=DEV)
    ws = torch.empty(tc.tc_copy_fragments_workspace(len(frags_np)), dtype=torch.uint8, device=DEV)
    dg = torch.empty(2 * len(frags_np), dtype=torch.int64, device=DEV)
    total = tc.tc_plan_fragments(frags, ws)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        # inputs produced on the side stream, consumed there without a sync
        src_flat.copy_(synth.random_bytes(src_flat.numel(), 63, device=DEV))
        tc.tc_gather_blocks(src, nb, B, B, ids, buf, stream=side)
        tc.tc_scatter_blocks(dst, nb, B, B, ids, buf, stream=side)
        fsrc.copy_(synth.random_bytes(fsrc.numel(), 64, device=DEV))
        tc.tc_copy_planned_digest(fsrc, fdst, ws, total, len(frags_np), dg, stream=side)
    side.synchronize()
    hs = [r.cpu().numpy() for r in src]
    want = oracle.gather_blocks(hs, B, B, ids_np)
    assert np.array_equal(buf.cpu().numpy(), want.reshape(-1))
    hd = [np.zeros(nb * B, np.uint8) for _ in range(R)]
    oracle.scatter_blocks(hd, B, B, ids_np, want.reshape(-1))
    assert np.array_equal(dst_flat.cpu().numpy(), np.concatenate(hd))
    hf = fsrc.cpu().numpy()
    wf = np.zeros(32 << 20, np.uint8)
    oracle.copy_fragments(hf, wf, frags_np)
    assert np.array_equal(fdst.cpu().numpy(), wf)
    assert np.array_equal(dg.cpu().numpy().view(np.uint64).reshape(-1, 2),
                          oracle.fragment_digests(hf, frags_np))


def _cast_items(rows, cols):
    """Two items over one ragged matrix: the top 256 rows (full tiles plus a
    partial right edge) and the rest (partial bottom tiles)."""
    tcn = (cols + 127) // 128
    items = np.zeros(2, dtype=tc.CAST_ITEM_DTYPE)
    items[0] = (0, 256, cols, cols, 0, cols, 0, tcn)
    items[1] = (256 * cols, rows - 256, cols, cols, 256 * cols, cols, 2 * tcn, tcn)
    return items


def test_graph_capture_and_replay():
    R, nb, B = 4, 256, 8192
    ids_np = synth.ids_without_replacement(nb, 100, seed=65)
    ids = torch.from_numpy(ids_np).to(DEV)
    src_flat, src = _pool(R, nb, B)
    dst_flat, dst = _pool(R, nb, B)
    buf = torch.empty(100 * R * B, dtype=torch.uint8, device=DEV)
    pool = 64 << 20
    frags_np = synth.fragment_storm(5000, pool, seed=66)      # unordered: a reordered plan
    frags = torch.from_numpy(frags_np.view(np.int64)).to(DEV)
    fsrc = torch.empty(pool, dtype=torch.uint8, device=DEV)
    fdst = torch.zeros(pool, dtype=torch.uint8, device=DEV)
    fdst2 = torch.zeros_like(fdst)
    fdst3 = torch.zeros_like(fdst)
    n = len(frags_np)
    wsb = tc.tc_copy_fragments_workspace(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    ws2 = torch.empty(wsb, dtype=torch.uint8, device=DEV)
    ws3 = torch.empty(tc.tc_copy_fragments_workspace_min(n), dtype=torch.uint8, device=DEV)
    dg = torch.empty(2 * n, dtype=torch.int64, device=DEV)
    x = torch.empty(65536 + 77, dtype=torch.bfloat16, device=DEV)
    q = torch.empty(x.numel(), dtype=torch.uint8, device=DEV)
    # block-scaled cast of a ragged matrix (one-call and planned) and its inverse
    rows, cols = 300, 520
    tcn = (cols + 127) // 128
    items = _cast_items(rows, cols)
    xc = torch.empty(rows * cols, dtype=torch.bfloat16, device=DEV)
    qc = torch.empty(rows * cols, dtype=torch.uint8, device=DEV)
    sc = torch.empty(3 * tcn, dtype=torch.float32, device=DEV)
    qp = torch.empty_like(qc)
    sp = torch.empty_like(sc)
    yc = torch.empty(rows * cols, dtype=torch.bfloat16, device=DEV)
    cws = torch.empty(tc.tc_cast_fp8_workspace(2), dtype=torch.uint8, device=DEV)
    pws = torch.empty_like(cws)
    dws = torch.empty(tc.tc_dequant_fp8_workspace(2), dtype=torch.uint8, device=DEV)
    ditems = items.astype(tc.DEQUANT_ITEM_DTYPE)       # same geometry, codes -> bf16
    # the planned cast and inverse with a per-tile table (workspace sized by items)
    qt, st = torch.empty_like(qc), torch.empty_like(sc)
    yt = torch.empty_like(yc)
    tws = torch.empty(tc.tc_cast_fp8_workspace_tiles(items), dtype=torch.uint8, device=DEV)
    tdws = torch.empty(tc.tc_dequant_fp8_workspace_tiles(ditems), dtype=torch.uint8, device=DEV)
    total = tc.tc_plan_fragments(frags, ws)
    plan = tc.tc_cast_fp8_prepare(xc, qp, items, pws)    # prepared eagerly, launched in the graph
    tplan = tc.tc_cast_fp8_prepare(xc, qt, items, tws)
    dplan = tc.tc_dequant_fp8_prepare(qt, yt, ditems, tdws)
    assert plan.tiled == 0 and tplan.tiled == 1 and dplan.tiled == 1
    assert tplan.full_tiles == dplan.full_tiles == 8    # the top 256 rows: 2 x 4 full tiles
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            s = torch.cuda.current_stream()
            tc.tc_gather_blocks(src, nb, B, B, ids, buf, stream=s)
            tc.tc_scatter_blocks(dst, nb, B, B, ids, buf, stream=s)
            tc.tc_copy_planned_digest(fsrc, fdst, ws, total, n, dg, stream=s)
            tc.tc_copy_planned(fsrc, fdst, ws, total, stream=s)
            tc.tc_copy_fragments(fsrc, fdst2, frags, ws2, stream=s)
            tc.tc_plan_fragments_async(frags, ws3, stream=s)     # the smallest workspace: larger pieces
            tc.tc_copy_planned(fsrc, fdst3, ws3, None, stream=s)
            tc.tc_cast_fp8_scaled(x, 0.25, q, stream=s)
            tc.tc_cast_fp8_blockscaled(xc, qc, sc, items, cws, stream=s)
            tc.tc_cast_fp8_planned(xc, qp, sp, pws, plan, stream=s)
            tc.tc_dequant_fp8_blockscaled(qc, sc, yc, ditems, dws, stream=s)
            tc.tc_cast_fp8_planned(xc, qt, st, tws, tplan, stream=s)
            tc.tc_dequant_fp8_planned(qt, st, yt, tdws, dplan, stream=s)
    torch.cuda.synchronize()
    # the graph holds its own copy of the item tables
    items[:] = np.zeros(1, dtype=tc.CAST_ITEM_DTYPE)
    ditems[:] = np.zeros(1, dtype=tc.DEQUANT_ITEM_DTYPE)
    want_items = _cast_items(rows, cols)

    for rep in range(4):
        # new inputs, written eagerly between replays
        src_flat.copy_(synth.random_bytes(src_flat.numel(), 70 + rep, device=DEV))
        fsrc.copy_(synth.random_bytes(fsrc.numel(), 80 + rep, device=DEV))
        x.copy_(synth.bf16_normal(x.numel(), 1.0, 90 + rep, device=DEV))
        xc.copy_(synth.bf16_normal(xc.numel(), 0.02 * (rep + 1), 95 + rep, device=DEV))
        dst_flat.zero_()
        fdst.zero_()
        fdst2.zero_()
        fdst3.zero_()
        dg.fill_(-1)
        for t in (qc, qp, qt):
            t.fill_(0xEE)
        for t in (sc, sp, st):
            t.fill_(-1.0)
        yc.zero_()
        yt.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        hs = [r.cpu().numpy() for r in src]
        want = oracle.gather_blocks(hs, B, B, ids_np)
        assert np.array_equal(buf.cpu().numpy(), want.reshape(-1)), rep
        hd = [np.zeros(nb * B, np.uint8) for _ in range(R)]
        oracle.scatter_blocks(hd, B, B, ids_np, want.reshape(-1))
        assert np.array_equal(dst_flat.cpu().numpy(), np.concatenate(hd)), rep
        hf = fsrc.cpu().numpy()
        wf = np.zeros(pool, np.uint8)
        oracle.copy_fragments(hf, wf, frags_np)
        assert np.array_equal(fdst.cpu().numpy(), wf), rep
        assert np.array_equal(fdst2.cpu().numpy(), wf), rep
        assert np.array_equal(fdst3.cpu().numpy(), wf), rep
        assert np.array_equal(dg.cpu().numpy().view(np.uint64).reshape(-1, 2),
                              oracle.fragment_digests(hf, frags_np)), rep
        xb = x.view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(q.cpu().numpy(), oracle.cast_fp8_scaled(xb, 0.25)), rep
        xcb = xc.view(torch.int16).cpu().numpy().view(np.uint16).reshape(rows, cols)
        wq_top, ws_top = oracle.cast_fp8_blockscaled(xcb[:256])
        wq_bot, ws_bot = oracle.cast_fp8_blockscaled(xcb[256:])
        wq = np.concatenate([wq_top, wq_bot])
        wsc = np.concatenate([ws_top.reshape(-1), ws_bot.reshape(-1)])
        for qq, ss in ((qc, sc), (qp, sp), (qt, st)):
            assert np.array_equal(qq.cpu().numpy().reshape(rows, cols), wq), rep
            assert np.array_equal(ss.cpu().numpy().view(np.uint32), wsc.view(np.uint32)), rep
        wy = np.concatenate([oracle.dequant_fp8_blockscaled(wq_top, ws_top),
                             oracle.dequant_fp8_blockscaled(wq_bot, ws_bot)])
        for yy in (yc, yt):
            assert np.array_equal(yy.view(torch.int16).cpu().numpy().view(np.uint16).reshape(rows, cols), wy), rep
    assert want_items.tobytes() != items.tobytes()


def test_concurrent_streams_independent_plans():
    """Three streams at once, none waiting for another: two planned copies
    with digests on their own workspaces (one plan reordered, one not) and a
    block gather.  Each result against the oracle."""
    pool = 64 << 20
    fa = synth.fragment_storm(6000, pool, seed=65)                   # unordered: reordered plan
    fb = fa[np.argsort(fa[:, 1], kind="stable")]                      # the same, ordered
    src = synth.random_bytes(pool, 66, device=DEV)
    outs, plans = [], []
    for fr in (fa, fb):
        frags = torch.from_numpy(fr.view(np.int64)).to(DEV)
        ws = torch.empty(tc.tc_copy_fragments_workspace(len(fr)), dtype=torch.uint8, device=DEV)
        plans.append((fr, ws, tc.tc_plan_fragments(frags, ws),
                      torch.zeros(pool, dtype=torch.uint8, device=DEV),
                      torch.empty(2 * len(fr), dtype=torch.int64, device=DEV)))
    R, nb, B = 4, 256, 32768
    ids_np = synth.ids_without_replacement(nb, 200, seed=67)
    ids = torch.from_numpy(ids_np).to(DEV)
    kv_flat, kv = _pool(R, nb, B)
    kv_flat.copy_(synth.random_bytes(kv_flat.numel(), 68, device=DEV))
    buf = torch.empty(200 * R * B, dtype=torch.uint8, device=DEV)
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in range(3)]
    for _ in range(3):                          # repeated, so the calls overlap in time
        for (fr, ws, total, dst, dg), st in zip(plans, streams):
            tc.tc_copy_planned_digest(src, dst, ws, total, len(fr), dg, stream=st)
        tc.tc_gather_blocks(kv, nb, B, B, ids, buf, stream=streams[2])
    for st in streams:
        st.synchronize()
    hsrc = src.cpu().numpy()
    for fr, ws, total, dst, dg in plans:
        want = np.zeros(pool, np.uint8)
        oracle.copy_fragments(hsrc, want, fr)
        assert np.array_equal(dst.cpu().numpy(), want)
        got = dg.cpu().numpy().view(np.uint64).reshape(-1, 2)
        assert np.array_equal(got, oracle.fragment_digests(hsrc, fr, use_src=True))
    want = oracle.gather_blocks([r.cpu().numpy() for r in kv], B, B, ids_np)
    assert np.array_equal(buf.cpu().numpy(), want.reshape(-1))
    assert int(plans[0][1][56:64].cpu().numpy().view(np.uint64)[0]) == 1   # reordered
    assert int(plans[1][1][56:64].cpu().numpy().view(np.uint64)[0]) == 0


def test_two_host_threads_cast_at_once():
    """Two host threads, each on its own stream, cast different item sets
    at the same time, over and over, each with its own workspace: nothing of
    one call's item table may leak into the other's (the tables travel in
    the launches' arguments; the library holds no shared buffer).  Every
    result against the oracle."""
    import threading
    rng = np.random.default_rng(131)
    jobs = []
    for k in range(2):
        rows, cols = 256 + 128 * k, 384 - 128 * k
        x = rng.normal(0, 0.02 * (k + 1), size=rows * cols).astype(np.float32)
        bits = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        # many small items: row bands of one tile row each, so the staged table is long
        items = np.zeros(rows // 128, dtype=tc.CAST_ITEM_DTYPE)
        for i in range(rows // 128):
            items[i] = (i * 128 * cols, 128, cols, cols, i * 128 * cols, cols,
                        i * ((cols + 127) // 128), (cols + 127) // 128)
        q_want, s_want = oracle.cast_fp8_blockscaled(bits.reshape(rows, cols))
        src = torch.from_numpy(bits.view(np.int16)).to(DEV)
        jobs.append(dict(src=src, items=items, rows=rows, cols=cols, q_want=q_want, s_want=s_want,
                         stream=torch.cuda.Stream(), errors=[]))

    def run(job):
        try:
            with torch.cuda.stream(job["stream"]):
                for _ in range(25):
                    q = torch.full((job["rows"] * job["cols"],), 0xEE, dtype=torch.uint8, device=DEV)
                    s = torch.full((s_len(job),), -1.0, dtype=torch.float32, device=DEV)
                    ws = torch.empty(tc.tc_cast_fp8_workspace(len(job["items"])), dtype=torch.uint8,
                                     device=DEV)
                    tc.tc_cast_fp8_blockscaled(job["src"], q, s, job["items"], ws, stream=job["stream"])
                    job["stream"].synchronize()
                    if not (np.array_equal(q.cpu().numpy().reshape(job["q_want"].shape), job["q_want"])
                            and np.array_equal(s.cpu().numpy().view(np.uint32),
                                               job["s_want"].reshape(-1).view(np.uint32))):
                        job["errors"].append("mismatch")
                        return
        except Exception as e:  # reported after the join
            job["errors"].append(repr(e))

    def s_len(job):
        return (job["rows"] // 128) * ((job["cols"] + 127) // 128)

    threads = [threading.Thread(target=run, args=(j,)) for j in jobs]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    assert [j["errors"] for j in jobs] == [[], []]
