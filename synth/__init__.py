"""Seeded synthetic inputs for the tensor-lifecycle data path.

This module is shared by the GPU path's tests and benchmark and by the CPU
oracle's tests.  It holds only input recipes -- shapes, id streams,
descriptor lists, permutations, random values -- and none of the arithmetic
of the operations themselves.

The inputs stand in for the paper's workloads, which use real models and
datasets that are not available here:

* KV block ids: requests re-using a popular prefix of paged KV blocks, as in
  the multi-turn agent workload of Sec. 6.4 and the KV reuse of Sec. 6.3
  (one Artifact per KV page).
* Model specs: weights of an 8B-shaped and a 70B-shaped dense transformer
  whose tensor-parallel slices are materialized per rank (Sec. 6.1, 6.2).
* Fragment storm: many small and large non-overlapping byte fragments, the
  high-cardinality tensor states of Sec. 4.2.
* MoE permutation: whole expert weights moved in a seeded expert order.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass

import numpy as np

GiB = 1 << 30
MiB = 1 << 20
KiB = 1 << 10

# ---------------------------------------------------------------------------
# Paged KV pools
# ---------------------------------------------------------------------------


@dataclass(frozen=True)
class KVShape:
    """Paged KV cache: one region per (layer, K|V), block-major inside it."""
    layers: int
    kv_heads: int
    head_dim: int
    block_tokens: int
    num_blocks: int
    n_ids: int
    elem_bytes: int = 2  # bf16

    @property
    def num_regions(self) -> int:
        return 2 * self.layers

    @property
    def block_bytes(self) -> int:
        return self.block_tokens * self.kv_heads * self.head_dim * self.elem_bytes

    @property
    def region_bytes(self) -> int:
        return self.num_blocks * self.block_bytes

    @property
    def transfer_bytes(self) -> int:
        return self.n_ids * self.num_regions * self.block_bytes


# 2 layers, K and V, 4 KV heads, head_dim 64, 16-token blocks, 256 blocks, 32 ids.
KV_TINY = KVShape(layers=2, kv_heads=4, head_dim=64, block_tokens=16, num_blocks=256, n_ids=32)
# Llama-3-8B-shaped: 32 layers, 8 KV heads, head_dim 128, 16-token blocks,
# 32768 blocks per region (1 GiB), 4096 ids per transfer.
KV_LLAMA3_8B = KVShape(layers=32, kv_heads=8, head_dim=128, block_tokens=16, num_blocks=32768, n_ids=4096)


def ids_without_replacement(num_blocks: int, n: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.choice(num_blocks, size=n, replace=False).astype(np.int32)


def ids_zipf_prefix_reuse(num_blocks: int, n: int, s: float, seed: int,
                          keep_duplicates: bool = False) -> np.ndarray:
    """Block ids of requests that re-use popular prefix blocks.

    A block's popularity rank k in [1, num_blocks] is drawn with
    P(k) ~ k^-s (truncated Zipf, inverse CDF on the cumulative weights) and
    mapped to a block id through a seeded permutation.  Draws continue until
    ``n`` distinct ids are seen; the ids are returned in first-occurrence
    order, so popular prefix blocks cluster at the front.  With
    ``keep_duplicates`` the first ``n`` raw draws are returned instead."""
    rng = np.random.default_rng(seed)
    perm = rng.permutation(num_blocks).astype(np.int32)
    w = np.arange(1, num_blocks + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    if keep_duplicates:
        ranks = np.searchsorted(cdf, rng.random(n), side="right")
        return perm[np.minimum(ranks, num_blocks - 1)]
    if n > num_blocks:
        raise ValueError("more distinct ids than blocks")
    out = []
    seen = np.zeros(num_blocks, dtype=bool)
    while len(out) < n:
        ranks = np.searchsorted(cdf, rng.random(max(4 * n, 1024)), side="right")
        ranks = np.minimum(ranks, num_blocks - 1)
        for k in ranks:
            if not seen[k]:
                seen[k] = True
                out.append(perm[k])
                if len(out) == n:
                    break
    return np.asarray(out, dtype=np.int32)


# ---------------------------------------------------------------------------
# Dense transformer weight specs (name, rows=out, cols=in, split)
# split: 'rows' = column-parallel (q, k, v, gate, up), 'cols' = row-parallel
# (o, down).  Layer-major stream order q, k, v, o, gate, up, down.
# ---------------------------------------------------------------------------


def dense_spec(layers: int, hidden: int, q_heads: int, kv_heads: int, head_dim: int, mlp: int):
    spec = []
    for l in range(layers):
        spec += [
            (f"l{l}.q", q_heads * head_dim, hidden, "rows"),
            (f"l{l}.k", kv_heads * head_dim, hidden, "rows"),
            (f"l{l}.v", kv_heads * head_dim, hidden, "rows"),
            (f"l{l}.o", hidden, q_heads * head_dim, "cols"),
            (f"l{l}.gate", mlp, hidden, "rows"),
            (f"l{l}.up", mlp, hidden, "rows"),
            (f"l{l}.down", hidden, mlp, "cols"),
        ]
    return spec


def spec_8b(layers: int = 32):
    """8B-shaped: q/o 4096x4096, k/v 1024x4096, gate/up 14336x4096, down 4096x14336."""
    return dense_spec(layers, hidden=4096, q_heads=32, kv_heads=8, head_dim=128, mlp=14336)


def spec_70b(layers: int = 80):
    """70B-shaped: hidden 8192, 64 q heads, 8 KV heads, head_dim 128, MLP 28672."""
    return dense_spec(layers, hidden=8192, q_heads=64, kv_heads=8, head_dim=128, mlp=28672)


def spec_scaled(layers: int, hidden: int, q_heads: int, kv_heads: int, head_dim: int, mlp: int):
    return dense_spec(layers, hidden, q_heads, kv_heads, head_dim, mlp)


def spec_elems(spec) -> int:
    return sum(r * c for (_, r, c, _) in spec)


# ---------------------------------------------------------------------------
# Fragment storm and MoE permutation: (src_off, dst_off, len) rows, uint64
# ---------------------------------------------------------------------------


def _layout(lens: np.ndarray, pool_bytes: int, align: int, rng) -> np.ndarray:
    """Place fragments of the given lengths in a pool in a random order with
    random gaps (multiples of ``align``) that use up the slack."""
    n = lens.size
    total = int(lens.sum())
    slack = pool_bytes - total
    if slack < 0:
        raise ValueError("fragments do not fit the pool")
    units = slack // align
    cuts = np.sort(rng.integers(0, units + 1, size=n, dtype=np.int64))
    gaps = np.diff(np.concatenate([[0], cuts])) * align  # gap before each placed fragment
    order = rng.permutation(n)
    placed_len = lens[order].astype(np.int64)
    starts = np.cumsum(gaps) + np.concatenate([[0], np.cumsum(placed_len)[:-1]])
    off = np.empty(n, dtype=np.int64)
    off[order] = starts
    return off


def fragment_storm(n: int, pool_bytes: int, seed: int, lo: int = 64, hi: int = 64 * KiB,
                   align: int = 16) -> np.ndarray:
    """``n`` fragments with log-uniform lengths in [lo, hi], rounded down to a
    multiple of ``align`` (at least ``lo``), laid out independently at random
    in a source pool and a destination pool.  ``align=1`` gives byte-granular
    offsets and lengths."""
    rng = np.random.default_rng(seed)
    lens = np.floor(np.exp(rng.uniform(np.log(lo), np.log(hi), size=n))).astype(np.int64)
    lens = np.maximum((lens // align) * align, lo)
    src = _layout(lens, pool_bytes, align, rng)
    dst = _layout(lens, pool_bytes, align, rng)
    return np.stack([src, dst, lens], axis=1).astype(np.uint64)


def fragment_mix(n: int, seed: int, align: int = 16, slack: float = 0.5, big_max: int = 4 * MiB):
    """``n`` fragments with mixed lengths -- about 10% empty, 20% tiny
    (below 64 bytes), 60% log-uniform in [64 B, 64 KiB], 10% large (up to
    ``big_max``) -- rounded down to multiples of ``align``, laid out at random in a
    source pool and a destination pool whose sizes exceed the payload by the
    fraction ``slack``.  Returns (rows, src_pool_bytes, dst_pool_bytes)."""
    rng = np.random.default_rng(seed)
    kind = rng.choice(4, size=n, p=[0.1, 0.2, 0.6, 0.1])
    lens = np.zeros(n, dtype=np.int64)
    tiny, mid, big = kind == 1, kind == 2, kind == 3
    lens[tiny] = rng.integers(1, 64, size=int(tiny.sum()))
    lens[mid] = np.floor(np.exp(rng.uniform(np.log(64), np.log(64 * KiB), size=int(mid.sum()))))
    lens[big] = rng.integers(64 * KiB, big_max, size=int(big.sum()))
    lens = (lens // align) * align
    total = int(lens.sum())
    pools = []
    for _ in range(2):
        pool = ((int(total * (1 + slack)) + 4096) // align + 1) * align
        pools.append(pool)
    src = _layout(lens, pools[0], align, rng)
    dst = _layout(lens, pools[1], align, rng)
    return np.stack([src, dst, lens], axis=1).astype(np.uint64), pools[0], pools[1]


def moe_permutation(n_experts: int, expert_bytes: int, seed: int):
    """Destination expert slot j receives source expert perm[j]."""
    rng = np.random.default_rng(seed)
    perm = rng.permutation(n_experts)
    j = np.arange(n_experts)
    frags = np.stack([perm * expert_bytes, j * expert_bytes,
                      np.full(n_experts, expert_bytes)], axis=1).astype(np.uint64)
    return frags, perm


# ---------------------------------------------------------------------------
# Values
# ---------------------------------------------------------------------------


def bf16_normal(numel: int, std: float, seed: int, device="cpu"):
    """bf16 N(0, std^2) values as a torch tensor (generated on ``device``)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    t = torch.empty(numel, dtype=torch.bfloat16, device=device)
    chunk = 1 << 28
    for s in range(0, numel, chunk):
        e = min(numel, s + chunk)
        t[s:e].normal_(0.0, std, generator=g)
    return t


def random_bytes(nbytes: int, seed: int, device="cpu"):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    t = torch.empty(nbytes, dtype=torch.uint8, device=device)
    chunk = 1 << 30
    for s in range(0, nbytes, chunk):
        e = min(nbytes, s + chunk)
        t[s:e].random_(0, 256, generator=g)
    return t


def sha256(a: np.ndarray) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


# Seeds: 1000 + config number for ids / descriptors and for values.
SEED_KV_TINY = 1001
SEED_KV_8B = 1002
SEED_RESHARD_8B = 1003
SEED_CAST_70B = 1004
SEED_STORM = 1005
