"""Pins for the oracle's bf16 -> E4M3 cast (CPU only).

The oracle is checked against things it does not compute itself:
  * reference points of the OCP E4M3 definition (tests/golden/e4m3_points.txt);
  * exact rational arithmetic (tests/exact.py): nearest-code search over all
    finite codes and a by-hand binary32 rounding of the quotient;
  * torch's float8_e4m3fn conversion, for finite |x| <= 448 (torch does not
    saturate, so larger inputs are outside what it can pin);
  * properties fixed by the mathematics: sign symmetry, monotonicity, the
    tile maximum mapping to +-448, the relative error bound.
"""
import math
import os
import struct
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from tests import exact

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e4m3_points.txt")

ALL_BF16 = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)


def _golden_points():
    pts = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            val, code = line.split()[:2]
            pts.append((val, int(code, 16)))
    return pts


@pytest.mark.parametrize("val,code", _golden_points())
def test_golden_points(val, code):
    x = float(np.float32(float(val)))
    if val.startswith("-") and x == 0:
        x = -0.0
    assert oracle.e4m3_encode(x) == code
    assert exact.encode_float(x) == code  # the exact reference agrees with the spec too


def test_decode_matches_definition_points():
    assert oracle.e4m3_decode(0x7E) == 448.0
    assert oracle.e4m3_decode(0x01) == 2.0 ** -9
    assert oracle.e4m3_decode(0x08) == 2.0 ** -6
    assert oracle.e4m3_decode(0x38) == 1.0
    assert oracle.e4m3_decode(0xFE) == -448.0
    assert math.isnan(oracle.e4m3_decode(0x7F)) and math.isnan(oracle.e4m3_decode(0xFF))
    for c in range(256):
        v = exact.e4m3_value(c)
        d = oracle.e4m3_decode(c)
        if v is None:
            assert math.isnan(d)
        else:
            assert Fraction(d) == v


def test_exhaustive_bf16_scale_one():
    """All 65536 bf16 patterns with scale 1 against exact nearest-code search."""
    got = oracle.cast_fp8_scaled(ALL_BF16, 1.0)
    want = np.array([exact.encode_float(exact.bf16_to_float(int(b))) for b in ALL_BF16],
                    dtype=np.uint8)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(hex(int(ALL_BF16[i])), hex(got[i]), hex(want[i])) for i in bad[:10]]


def test_torch_float8_agrees_in_range():
    """torch's CPU float8_e4m3fn conversion as a third opinion, finite |x| <= 448."""
    x = torch.from_numpy(ALL_BF16.view(np.int16)).view(torch.bfloat16)
    f = x.float()
    keep = torch.isfinite(f) & (f.abs() <= 448)
    ref = f[keep].to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = oracle.cast_fp8_scaled(ALL_BF16[keep.numpy()], 1.0)
    assert np.array_equal(got, ref)


def _random_scales(rng, n):
    """Scales across the binary32 range: normal, powers of two, subnormal."""
    bits = rng.integers(0x00800000, 0x7F000000, size=n, dtype=np.int64)
    sub = rng.integers(1, 0x00800000, size=n // 8, dtype=np.int64)
    pow2 = (np.arange(-20, 21) + 127) << 23
    allb = np.concatenate([bits, sub, pow2]).astype(np.uint32)
    return allb.view(np.float32)


def test_scaled_quotient_against_exact_rounding():
    """q = enc(RN_f32(x / s)) checked with exact rational division."""
    rng = np.random.default_rng(7)
    scales = _random_scales(rng, 64)
    for s in scales:
        s = float(s)
        xb = rng.integers(0, 1 << 16, size=300, dtype=np.int64).astype(np.uint16)
        got = oracle.cast_fp8_scaled(xb, s)
        for b, g in zip(xb, got):
            x = exact.bf16_to_float(int(b))
            if math.isnan(x):
                want = 0x7F
            elif math.isinf(x):
                want = exact.encode_float(x / s)
            else:
                want = exact.quotient_code(x, s)
            assert g == want, (hex(int(b)), s, hex(g), hex(want))


def test_quotients_near_every_midpoint():
    """Quotients placed within a few binary32 ulps of every E4M3 rounding
    midpoint: the double rounding (binary32 first, then E4M3) must match
    the exact reference on both sides of each midpoint."""
    vals = [v for v, _ in exact._POS]
    mids = [(a + b) / 2 for a, b in zip(vals[:-1], vals[1:])] + [Fraction(464)]
    rng = np.random.default_rng(11)
    # choose x in bf16 and s = x / target so that x / s lands near the midpoint
    for m in mids:
        if m == 0:
            continue
        mf = exact.bits_f32(exact.f32_bits(float(m)))
        for delta in (-3, -2, -1, 0, 1, 2, 3):
            target = exact.bits_f32(exact.f32_bits(mf) + delta)
            xb = int(rng.integers(0x3F80, 0x4000))  # x in [1, 2)
            x = exact.bf16_to_float(xb)
            s = float(np.float32(x / target))
            if s == 0 or not math.isfinite(s):
                continue
            got = oracle.cast_fp8_scaled(np.array([xb], dtype=np.uint16), s)[0]
            assert got == exact.quotient_code(x, s), (float(m), delta, x, s)


def test_sign_symmetry_and_monotonicity():
    pos = ALL_BF16[ALL_BF16 < 0x7F80]           # +0 .. largest finite
    neg = pos | np.uint16(0x8000)
    qp = oracle.cast_fp8_scaled(pos, 0.75)
    qn = oracle.cast_fp8_scaled(neg, 0.75)
    assert np.array_equal(qn, qp | 0x80)
    # decoded values are non-decreasing in x for x >= 0 (bf16 bit order = value order)
    dec = np.array([oracle.e4m3_decode(int(c)) for c in qp])
    assert np.all(np.diff(dec) >= 0)


def test_special_inputs_scaled():
    sp = np.array([0x7F80, 0xFF80, 0x7FC0, 0xFFC1, 0x0000, 0x8000], dtype=np.uint16)
    got = oracle.cast_fp8_scaled(sp, 1.0)
    assert list(got) == [0x7E, 0xFE, 0x7F, 0x7F, 0x00, 0x80]


# ---------------------------------------------------------------------------
# block-scaled cast
# ---------------------------------------------------------------------------

def _bits_from_float(a: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of float32 values (round to nearest even)."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _exact_blockscaled(xb: np.ndarray):
    """Reference for one matrix with exact rationals, tile by tile."""
    rows, cols = xb.shape
    tr, tc = (rows + 127) // 128, (cols + 127) // 128
    q = np.zeros((rows, cols), dtype=np.uint8)
    s = np.zeros((tr, tc), dtype=np.uint32)
    for ti in range(tr):
        for tj in range(tc):
            blk = xb[ti * 128:(ti + 1) * 128, tj * 128:(tj + 1) * 128]
            vals = [exact.bf16_to_float(int(b)) for b in blk.reshape(-1)]
            if any(not math.isfinite(v) for v in vals):
                s[ti, tj] = 0x7FC00000
                q[ti * 128:(ti + 1) * 128, tj * 128:(tj + 1) * 128] = 0x7F
                continue
            amax = max(Fraction(abs(v)) for v in vals)
            if amax == 0:
                s[ti, tj] = 0
                q[ti * 128:(ti + 1) * 128, tj * 128:(tj + 1) * 128] = np.where(blk & 0x8000, 0x80, 0)
                continue
            sc = exact.rn_f32(amax / 448)
            s[ti, tj] = exact.f32_bits(sc)
            codes = [exact.quotient_code(v, sc) for v in vals]
            q[ti * 128:(ti + 1) * 128, tj * 128:(tj + 1) * 128] = np.array(codes, dtype=np.uint8).reshape(blk.shape)
    return q, s


def test_blockscaled_exact_small_ragged():
    rng = np.random.default_rng(3)
    a = rng.normal(0, 0.02, size=(150, 260)).astype(np.float32)
    a[140:150, 200:210] *= 1e-3                 # a quiet corner inside an edge tile
    xb = _bits_from_float(a)
    q, s = oracle.cast_fp8_blockscaled(xb)
    qe, se = _exact_blockscaled(xb)
    assert np.array_equal(s.view(np.uint32), se)
    assert np.array_equal(q, qe)


def test_blockscaled_special_tiles():
    rng = np.random.default_rng(5)
    a = rng.normal(0, 1, size=(256, 512)).astype(np.float32)
    a[0:128, 0:128] = 0.0                       # all-zero tile
    a[0:128, 0:128][::3, ::5] = -0.0            # with some negative zeros
    a[0:128, 128:256][7, 9] = np.inf            # Inf tile
    a[0:128, 256:384][100, 1] = np.nan          # NaN tile
    a[128:256, 0:128] *= 1e-38                  # bf16 subnormal amax -> subnormal scale
    a[128:256, 128:256] = 0.0
    a[128:256, 128:256][5, 5] = 2.0 ** -133     # smallest bf16 subnormal as amax
    a[128:256, 128:256][6, 6] = -(2.0 ** -133)
    xb = _bits_from_float(a)
    q, s = oracle.cast_fp8_blockscaled(xb)
    qe, se = _exact_blockscaled(xb)
    assert np.array_equal(s.view(np.uint32), se)
    assert np.array_equal(q, qe)
    assert s.view(np.uint32)[0, 1] == 0x7FC00000 and np.all(q[0:128, 128:256] == 0x7F)
    assert s[0, 0] == 0.0 and set(np.unique(q[0:128, 0:128])) <= {0x00, 0x80}
    assert 0 < s[1, 0] < np.finfo(np.float32).tiny   # subnormal scale kept, not flushed
    assert q[128 + 5, 128 + 5] == 0x7E and q[128 + 6, 128 + 6] == 0xFE


def test_blockscaled_invariants():
    """Per tile: the element of largest magnitude encodes to +-448; every
    element reconstructs within the E4M3 rounding bound; strided source view
    gives the same answer as a packed copy."""
    rng = np.random.default_rng(9)
    full = _bits_from_float(rng.normal(0, 0.02, size=(384, 1024)).astype(np.float32))
    view = full[:, 256:640]                     # a column slice, row stride 1024
    q, s = oracle.cast_fp8_blockscaled(view)
    q2, s2 = oracle.cast_fp8_blockscaled(np.ascontiguousarray(view))
    assert np.array_equal(q, q2) and np.array_equal(s, s2)
    x = torch.from_numpy(np.ascontiguousarray(view).view(np.int16)).view(torch.bfloat16).float().numpy()
    dec = np.vectorize(oracle.e4m3_decode)(q).astype(np.float64)
    for ti in range(3):
        for tj in range(3):
            xs = x[ti * 128:(ti + 1) * 128, tj * 128:(tj + 1) * 128].astype(np.float64)
            qs = q[ti * 128:(ti + 1) * 128, tj * 128:(tj + 1) * 128]
            k = np.unravel_index(np.argmax(np.abs(xs)), xs.shape)
            assert qs[k] == (0xFE if xs[k] < 0 else 0x7E)
            sc = float(s[ti, tj])
            rec = dec[ti * 128:(ti + 1) * 128, tj * 128:(tj + 1) * 128] * sc
            err = np.abs(rec - xs)
            normal = np.abs(xs) / sc >= 2.0 ** -6
            bound = np.where(normal, (2.0 ** -4 + 2.0 ** -23) * np.abs(xs),
                             2.0 ** -10 * sc + 2.0 ** -23 * np.abs(xs))
            assert np.all(err <= bound * (1 + 1e-12))


# ---------------------------------------------------------------------------
# inverse cast: E4M3 + tile scale -> bf16
# ---------------------------------------------------------------------------

def _dequant_exact(code: int, s: float) -> int:
    v = exact.e4m3_value(code)
    if v is None or math.isnan(s):
        return 0x7FC0
    if math.isinf(s):
        if v == 0:
            return 0x7FC0                     # 0 * Inf
        neg = (v < 0) != (s < 0)
        return (0x8000 if neg else 0) | 0x7F80
    prod = Fraction(v) * Fraction(s)
    neg_zero = prod == 0 and ((code & 0x80) != 0) != (math.copysign(1.0, s) < 0)
    return exact.rn_bf16_of_f32(exact.rn_f32(prod, negative_zero=neg_zero))


def test_dequant_every_code_at_many_scales():
    rng = np.random.default_rng(60)
    scales = list(_random_scales(rng, 24)) + [0.0, -0.0, 1.0, 2.0 ** -140, 3.4e38, float("inf"),
                                              float("nan")]
    codes = np.arange(256, dtype=np.uint8)
    for s in scales:
        s32 = float(np.float32(s))
        q = np.tile(codes, 128).reshape(128, 256)
        sg = np.full((1, 2), s32, dtype=np.float32)
        y = oracle.dequant_fp8_blockscaled(q, sg)
        want = np.array([_dequant_exact(int(c), s32) for c in codes], dtype=np.uint16)
        assert np.array_equal(y[0], want), s32
        assert np.array_equal(y[77], want)


def test_dequant_matches_torch_for_finite_results():
    """torch: float8_e4m3fn -> float32, times the scale, -> bfloat16 (RNE)."""
    rng = np.random.default_rng(61)
    q = rng.integers(0, 256, size=(256, 384), dtype=np.int64).astype(np.uint8)
    s = (rng.uniform(0.5, 2.0, size=(2, 3)) * 10.0 ** rng.integers(-30, 30, size=(2, 3))).astype(np.float32)
    y = oracle.dequant_fp8_blockscaled(q, s)
    t = torch.from_numpy(q).view(torch.float8_e4m3fn).float()
    tiles = torch.from_numpy(np.repeat(np.repeat(s, 128, axis=0), 128, axis=1))
    ref = (t * tiles).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    finite = np.isfinite((t * tiles).numpy())
    assert np.array_equal(y[finite], ref[finite])


def test_dequant_inverts_the_cast_within_the_rounding_bound():
    rng = np.random.default_rng(62)
    a = rng.normal(0, 0.02, size=(300, 260)).astype(np.float32)
    xb = _bits_from_float(a)
    q, s = oracle.cast_fp8_blockscaled(xb)
    y = oracle.dequant_fp8_blockscaled(q, s)
    x = torch.from_numpy(xb.view(np.int16)).view(torch.bfloat16).float().numpy().astype(np.float64)
    back = torch.from_numpy(y.view(np.int16)).view(torch.bfloat16).float().numpy().astype(np.float64)
    scale_el = np.repeat(np.repeat(s.astype(np.float64), 128, axis=0), 128, axis=1)[:300, :260]
    normal = np.abs(x) / scale_el >= 2.0 ** -6
    # E4M3 relative error 2^-4, then bf16 rounding 2^-9 of the result
    bound = np.where(normal, (2.0 ** -4) * np.abs(x), 2.0 ** -10 * scale_el) * (1 + 2.0 ** -8) + \
        2.0 ** -9 * np.abs(back)
    assert np.all(np.abs(back - x) <= bound)


def test_bf16_rounding_matches_torch():
    """The oracle's binary32 -> bf16 step of the inverse against torch's
    float32 -> bfloat16 conversion (nearest, ties to even): random patterns,
    exact ties and their neighbours at many exponents, subnormals, the
    largest finite values, the overflow boundary and infinities; NaN gives
    the canonical 0x7FC0."""
    rng = np.random.default_rng(63)
    pats = [rng.integers(0, 1 << 32, size=20000, dtype=np.uint64)]
    mant = rng.integers(0, 1 << 7, size=400, dtype=np.uint64) << np.uint64(16)
    for e in list(range(0, 6)) + list(range(100, 140)) + list(range(248, 256)):
        base = (np.uint64(e) << np.uint64(23)) | mant
        for d in (0x7FFF, 0x8000, 0x8001, 0x18000, 0xFFFF):      # below, at, above a tie; odd-LSB tie
            pats.append(base | np.uint64(d & 0xFFFF) | (np.uint64(d >> 16) << np.uint64(16)))
    pats.append(np.array([0x7F7F7FFF, 0x7F7F8000, 0x7F7FFFFF, 0x7F800000, 0x00000001, 0x007FFFFF,
                          0x00008000, 0x00018000], dtype=np.uint64))
    bits = np.concatenate(pats) & np.uint64(0xFFFFFFFF)
    bits = np.concatenate([bits, bits | np.uint64(0x80000000)]).astype(np.uint32)
    vals = bits.view(np.float32)
    finite_or_inf = ~np.isnan(vals)
    ref = torch.from_numpy(vals.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([oracle.bf16_round(float(v)) for v in vals], dtype=np.uint16)
    assert np.array_equal(got[finite_or_inf], ref[finite_or_inf])
    assert np.all(got[~finite_or_inf] == 0x7FC0)
