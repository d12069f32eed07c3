"""GPU parity: paged-KV block gather (publish) and scatter (hydrate).

The HIP path (through the C ABI) against the CPU oracle, byte for byte, on
the same seeded inputs; full-size Llama-3-8B-shaped pools are checked on
sampled blocks against the oracle and, for every block, by properties.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
import paper_2608_06007_amd as tc

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _host(t):
    return t.detach().to("cpu").numpy()


def _regions_random(R, nb, B, stride, seed):
    g = torch.Generator(device=DEV)
    g.manual_seed(seed)
    span = (nb - 1) * stride + B
    return [torch.randint(0, 256, (span,), dtype=torch.uint8, device=DEV, generator=g) for _ in range(R)]


def _run_pair(regions, nb, B, stride, ids_np, sentinel=0xA5):
    """GPU gather + scatter into a sentinel pool, and the same with the oracle."""
    R = len(regions)
    ids = torch.from_numpy(ids_np.astype(np.int32)).to(DEV)
    out = torch.empty(len(ids_np) * R * B, dtype=torch.uint8, device=DEV)
    tc.tc_gather_blocks(regions, nb, B, stride, ids, out)
    dst = [torch.full_like(r, sentinel) for r in regions]
    tc.tc_scatter_blocks(dst, nb, B, stride, ids, out)
    torch.cuda.synchronize()
    host_src = [_host(r) for r in regions]
    want = oracle.gather_blocks(host_src, B, stride, ids_np)
    assert np.array_equal(_host(out).reshape(want.shape), want)
    host_dst = [np.full_like(h, sentinel) for h in host_src]
    oracle.scatter_blocks(host_dst, B, stride, ids_np, want)
    for d, h in zip(dst, host_dst):
        assert np.array_equal(_host(d), h)


def test_tiny_config():
    """2 layers x K/V, 4 heads, dim 64, 16-token blocks, 256 blocks, 32 ids."""
    s = synth.KV_TINY
    vals = synth.bf16_normal(s.num_regions * s.region_bytes // 2, 1.0, synth.SEED_KV_TINY, device=DEV)
    flat = vals.view(torch.uint8)
    regions = [flat[r * s.region_bytes:(r + 1) * s.region_bytes] for r in range(s.num_regions)]
    ids = synth.ids_without_replacement(s.num_blocks, s.n_ids, synth.SEED_KV_TINY)
    _run_pair(regions, s.num_blocks, s.block_bytes, s.block_bytes, ids)


@pytest.mark.parametrize("B,stride", [(8192, 8192), (8192 + 16, 8192 + 48), (100, 104), (16, 16),
                                      (40000, 40960), (3, 7)])
def test_block_geometries(B, stride):
    nb = 40
    regions = _regions_random(3, nb, B, stride, 7)
    ids = synth.ids_without_replacement(nb, 25, seed=8)
    _run_pair(regions, nb, B, stride, ids)


def test_every_small_block_size_and_stride_pad():
    """Block sizes 1 .. 48 bytes and 4080 .. 4112 (around the 4 KiB tile), each
    with stride pads 0, 1, 15 and 16: the byte path and the vector path's
    tiles and tails, through gather and scatter, against the oracle."""
    nb = 12
    ids = synth.ids_without_replacement(nb, 7, seed=12)
    for B in list(range(1, 49)) + list(range(4080, 4113)):
        for pad in (0, 1, 15, 16):
            regions = _regions_random(2, nb, B, B + pad, 13 + B + pad)
            _run_pair(regions, nb, B, B + pad, ids)


def test_edge_ids():
    nb, B = 64, 4096
    regions = _regions_random(4, nb, B, B, 9)
    _run_pair(regions, nb, B, B, np.array([nb - 1], dtype=np.int32))        # single, max id
    _run_pair(regions, nb, B, B, np.arange(nb, dtype=np.int32))             # all ids: plain copy
    _run_pair(regions, nb, B, B, np.array([0], dtype=np.int32))


def test_gather_repeated_ids_and_empty():
    nb, B = 16, 2048
    regions = _regions_random(2, nb, B, B, 10)
    ids_np = np.array([5, 5, 1, 5], dtype=np.int32)
    ids = torch.from_numpy(ids_np).to(DEV)
    out = torch.empty(4 * 2 * B, dtype=torch.uint8, device=DEV)
    tc.tc_gather_blocks(regions, nb, B, B, ids, out)
    torch.cuda.synchronize()
    want = oracle.gather_blocks([_host(r) for r in regions], B, B, ids_np)
    assert np.array_equal(_host(out).reshape(want.shape), want)
    empty = torch.empty(0, dtype=torch.int32, device=DEV)
    tc.tc_gather_blocks(regions, nb, B, B, empty, out)        # n = 0: nothing happens
    tc.tc_scatter_blocks(regions, nb, B, B, empty, out)


def test_binding_refuses_host_and_strided_tensors():
    """The library addresses every buffer as one flat device byte range, so
    the binding refuses host tensors and non-contiguous views before any
    launch (a strided view's flat range would reach past the view)."""
    nb, B = 8, 256
    regions = _regions_random(2, nb, B, B, 11)
    ids = torch.tensor([1, 3], dtype=torch.int32, device=DEV)
    out = torch.empty(2 * 2 * B, dtype=torch.uint8, device=DEV)
    with pytest.raises(ValueError):
        tc.tc_gather_blocks(regions, nb, B, B, ids, out.cpu())
    strided = torch.empty(2 * 2 * B * 2, dtype=torch.uint8, device=DEV)[::2]
    with pytest.raises(ValueError):
        tc.tc_gather_blocks(regions, nb, B, B, ids, strided)
    with pytest.raises(ValueError):
        tc.tc_gather_blocks(regions, nb, B, B, torch.tensor([1, 0, 3, 0], dtype=torch.int32,
                                                            device=DEV)[::2], out)
    with pytest.raises(ValueError):                          # the library reads int32 ids
        tc.tc_gather_blocks(regions, nb, B, B, ids.to(torch.int64), out)
    tc.tc_gather_blocks(regions, nb, B, B, ids, out)         # the same call, contiguous
    torch.cuda.synchronize()


def test_interleaved_engine_layout():
    """One allocation laid out [blocks][2][...]: K and V of a layer are two
    regions with base offset block_bytes apart and stride 2*block_bytes."""
    nb, B = 32, 1024
    layers = 3
    g = torch.Generator(device=DEV)
    g.manual_seed(11)
    allocs = [torch.randint(0, 256, (nb * 2 * B,), dtype=torch.uint8, device=DEV, generator=g)
              for _ in range(layers)]
    regions = []
    for a in allocs:
        regions += [a.data_ptr(), a.data_ptr() + B]
    ids_np = synth.ids_without_replacement(nb, 12, seed=12)
    ids = torch.from_numpy(ids_np).to(DEV)
    out = torch.empty(12 * 2 * layers * B, dtype=torch.uint8, device=DEV)
    tc.tc_gather_blocks(regions, nb, B, 2 * B, ids, out)
    dst_allocs = [torch.full_like(a, 0x33) for a in allocs]
    dst_regions = []
    for a in dst_allocs:
        dst_regions += [a.data_ptr(), a.data_ptr() + B]
    tc.tc_scatter_blocks(dst_regions, nb, B, 2 * B, ids, out)
    torch.cuda.synchronize()
    host = []
    for a in allocs:
        h = _host(a)
        host += [h[:(nb - 1) * 2 * B + B], h[B:]]
    want = oracle.gather_blocks(host, B, 2 * B, ids_np)
    assert np.array_equal(_host(out).reshape(want.shape), want)
    for a, d in zip(allocs, dst_allocs):
        av, dv = _host(a).reshape(nb, 2 * B), _host(d).reshape(nb, 2 * B)
        mask = np.zeros(nb, dtype=bool)
        mask[ids_np] = True
        assert np.array_equal(dv[mask], av[mask]) and np.all(dv[~mask] == 0x33)


def test_validation_mode_reports_bad_ids():
    nb, B = 8, 256
    regions = _regions_random(2, nb, B, B, 13)
    out = torch.empty(2 * 2 * B, dtype=torch.uint8, device=DEV)
    tc.tc_set_validate(True)
    try:
        with pytest.raises(tc.TcError) as e:
            tc.tc_gather_blocks(regions, nb, B, B, torch.tensor([0, 8], dtype=torch.int32, device=DEV), out)
        assert e.value.status == 2
        with pytest.raises(tc.TcError) as e:
            tc.tc_scatter_blocks(regions, nb, B, B, torch.tensor([3, 3], dtype=torch.int32, device=DEV), out)
        assert e.value.status == 3
        # a good call still works with validation on
        tc.tc_gather_blocks(regions, nb, B, B, torch.tensor([1, 2], dtype=torch.int32, device=DEV), out)
        torch.cuda.synchronize()
    finally:
        tc.tc_set_validate(False)


def test_llama3_8b_full_size():
    """32 layers x K/V, 8 heads, dim 128, 16-token blocks, 32768 blocks per
    region (64 GiB per pool), 4096 Zipf(1.1) ids: the benchmark's workload."""
    s = synth.KV_LLAMA3_8B
    B, nb, R = s.block_bytes, s.num_blocks, s.num_regions
    try:
        _full_size_body(s, B, nb, R)
    finally:
        torch.cuda.synchronize()


def _full_size_body(s, B, nb, R):
    pool_a = synth.bf16_normal(R * s.region_bytes // 2, 1.0, synth.SEED_KV_8B, device=DEV).view(torch.uint8)
    regions_a = [pool_a[r * s.region_bytes:(r + 1) * s.region_bytes] for r in range(R)]
    ids_np = synth.ids_zipf_prefix_reuse(nb, s.n_ids, 1.1, synth.SEED_KV_8B)
    ids = torch.from_numpy(ids_np).to(DEV)
    buf = torch.empty(s.transfer_bytes, dtype=torch.uint8, device=DEV)
    tc.tc_gather_blocks(regions_a, nb, B, B, ids, buf)
    pool_b = torch.full((R * s.region_bytes,), 0xA5, dtype=torch.uint8, device=DEV)
    regions_b = [pool_b[r * s.region_bytes:(r + 1) * s.region_bytes] for r in range(R)]
    tc.tc_scatter_blocks(regions_b, nb, B, B, ids, buf)
    torch.cuda.synchronize()
    bufv = buf.view(s.n_ids, R, B)
    # every chunk against the oracle, one region at a time (64 passes over a
    # 1 GiB host copy of the region): the gathered blocks, and the hydrated
    # region of pool B (the oracle's scatter into a sentinel region)
    for r in range(R):
        print(f"region {r}", flush=True) if r % 16 == 0 else None
        host_a = _host(regions_a[r])
        want = oracle.gather_blocks([host_a], B, B, ids_np)
        assert np.array_equal(_host(bufv[:, r].contiguous()), want[:, 0, :]), r
        want_b = np.full(s.region_bytes, 0xA5, dtype=np.uint8)
        oracle.scatter_blocks([want_b], B, B, ids_np, want.reshape(-1))
        assert np.array_equal(_host(regions_b[r]), want_b), r
    # and every block against torch.index_select on the device
    idl = ids.long()
    for r in range(R):
        a = regions_a[r].view(nb, B)
        assert torch.equal(torch.index_select(a, 0, idl), bufv[:, r])


def test_region_larger_than_4gib():
    """One region of 100,000 blocks of 64 KiB (6.55 GB): block addresses past
    2^32, ids at both ends of the region."""
    nb, B = 100_000, 65536
    region = synth.random_bytes(nb * B, 48, device=DEV)
    ids_np = np.array([nb - 1, 0, 65536, 65535, nb - 2, 70000], dtype=np.int32)
    ids = torch.from_numpy(ids_np).to(DEV)
    buf = torch.empty(len(ids_np) * B, dtype=torch.uint8, device=DEV)
    tc.tc_gather_blocks([region], nb, B, B, ids, buf)
    torch.cuda.synchronize()
    for k, i in enumerate(ids_np):
        want = oracle.gather_blocks([_host(region[int(i) * B:(int(i) + 1) * B])], B, B,
                                    np.array([0], np.int32))
        assert np.array_equal(_host(buf[k * B:(k + 1) * B]), want.reshape(-1)), int(i)
    # scatter them back shifted by one slot, then gather again
    ids2 = torch.from_numpy(np.array([1, 2, 3, 4, 5, 6], np.int32)).to(DEV)
    tc.tc_scatter_blocks([region], nb, B, B, ids2, buf)
    back = torch.empty_like(buf)
    tc.tc_gather_blocks([region], nb, B, B, ids2, back)
    torch.cuda.synchronize()
    assert torch.equal(back, buf)
    del region
    torch.cuda.empty_cache()


def test_more_tiles_than_one_grid_holds():
    """2^24 + 5 one-tile chunks (16-byte blocks, one region): more workgroup
    tiles than one launch's grid takes, so the grid strides, and enough that a
    grid of one workgroup per tile would not fit a dispatch's 32-bit count of
    work-items.  Byte for byte against the oracle, gather and scatter."""
    n = (1 << 24) + 5
    B = 16
    nb = n + 11
    region = synth.random_bytes(nb * B, 131, device=DEV)
    ids_np = np.random.default_rng(131).permutation(nb)[:n].astype(np.int32)
    ids = torch.from_numpy(ids_np).to(DEV)
    buf = torch.empty(n * B, dtype=torch.uint8, device=DEV)
    tc.tc_gather_blocks([region], nb, B, B, ids, buf)
    dst = torch.full_like(region, 0x5A)
    tc.tc_scatter_blocks([dst], nb, B, B, ids, buf)
    torch.cuda.synchronize()
    host = _host(region)
    want = oracle.gather_blocks([host], B, B, ids_np)
    assert np.array_equal(_host(buf).reshape(want.shape), want)
    back = np.full_like(host, 0x5A)
    oracle.scatter_blocks([back], B, B, ids_np, want)
    assert np.array_equal(_host(dst), back)
    del region, dst, buf
    torch.cuda.empty_cache()
