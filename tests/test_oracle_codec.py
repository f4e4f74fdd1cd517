"""Pins of the oracle's blockwise absmax codec (App. B.1, Eq. fp8-roundtrip,
in the scaled reading: one fp32 scale per 1 x block run of a row).

Each pin is fixed by something other than the oracle's own code: exact
round trips of values already on the code grid, the exact rational quotient
rounded by brute-force enumeration of the code grid, error bounds that follow
from the formats, and torch's casts.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

from paper_2609_33570_amd import workloads as wl

Q = {0: 127, 1: 448}


def e4m3_grid():
    """Finite non-negative E4M3FN values and their codes, by definition."""
    out = []
    for e in range(16):
        for m in range(8):
            if e == 15 and m == 7:
                continue
            v = Fraction(m, 512) if e == 0 else (1 + Fraction(m, 8)) * Fraction(2) ** (e - 7)
            out.append((v, (e << 3) | m))
    return out


E4M3 = e4m3_grid()


def bits(x):
    return wl.to_bf16_bits(np.asarray(x, dtype=np.float32))


def f32(bf):
    return (np.asarray(bf, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@pytest.mark.parametrize("block", [32, 64, 128, 256])
def test_grid_roundtrip_int8(orc, block):
    g = np.random.default_rng(1)
    rows, nb = 6, 5
    q = g.integers(-127, 128, size=(rows, nb, block))
    pos = g.integers(0, block, size=(rows, nb))
    sign = np.where(g.random((rows, nb)) < 0.5, -1, 1)
    np.put_along_axis(q, pos[..., None], (127 * sign)[..., None], axis=2)
    k = g.integers(-30, 30, size=(rows, nb))
    x = (q * np.exp2(k)[..., None]).reshape(rows, nb * block).astype(np.float32)
    xb = bits(x)
    assert np.array_equal(f32(xb), x)  # on the bf16 grid
    codes, scales = orc.quantize(xb, orc.INT8, block)
    assert np.array_equal(codes.view(np.int8).astype(np.int64), q.reshape(rows, -1))
    assert np.array_equal(scales, np.exp2(k).astype(np.float32))
    xh = orc.dequantize(codes, scales, orc.INT8, block)
    assert np.array_equal(f32(xh), x)


@pytest.mark.parametrize("block", [32, 128])
def test_grid_roundtrip_e4m3(orc, block):
    g = np.random.default_rng(2)
    rows, nb = 6, 5
    vals = np.array([float(v) for v, _ in E4M3])
    codes_of = np.array([c for _, c in E4M3], dtype=np.uint8)
    idx = g.integers(0, len(vals), size=(rows, nb, block))
    sgn = g.random((rows, nb, block)) < 0.5
    pos = g.integers(0, block, size=(rows, nb))
    np.put_along_axis(idx, pos[..., None], len(vals) - 1, axis=2)  # 448 somewhere
    k = g.integers(-20, 20, size=(rows, nb))
    v = np.where(sgn, -vals[idx], vals[idx])
    x = (v * np.exp2(k)[..., None]).reshape(rows, -1).astype(np.float32)
    expect = (codes_of[idx] | np.where(sgn, 0x80, 0)).reshape(rows, -1).astype(np.uint8)
    xb = bits(x)
    assert np.array_equal(f32(xb), x)
    codes, scales = orc.quantize(xb, orc.E4M3FN, block)
    assert np.array_equal(codes, expect)
    assert np.array_equal(scales, np.exp2(k).astype(np.float32))
    xh = orc.dequantize(codes, scales, orc.E4M3FN, block)
    assert np.array_equal(xh, xb)  # bit for bit, sign of zero included


@pytest.mark.parametrize("code", [0, 1])
def test_block_max_encodes_to_full_scale(orc, code):
    x = wl.activation_host(64, 512, seed=5, outliers=("entries", 0.01, 20.0))
    codes, scales = orc.quantize(x, code, 64)
    xf = np.abs(f32(x)).reshape(64, 8, 64)
    arg = xf.argmax(axis=2)
    c = np.take_along_axis(codes.reshape(64, 8, 64), arg[..., None], axis=2)[..., 0]
    full = {0: (0x7F, 0x81), 1: (0x7E, 0xFE)}[code]
    assert np.isin(c, full).all()


def _nearest_int_even(v: Fraction) -> int:
    fl = v.numerator // v.denominator
    frac = v - fl
    if frac > Fraction(1, 2):
        return fl + 1
    if frac < Fraction(1, 2):
        return fl
    return fl if fl % 2 == 0 else fl + 1


def _nearest_e4m3(v: Fraction) -> int:
    a = abs(v)
    best = None
    for gv, c in E4M3:
        d = abs(gv - a)
        if best is None or d < best[0] or (d == best[0] and (c & 1) == 0):
            best = (d, c)
    return best[1] | (0x80 if v < 0 else 0)


def _near_tie(v: Fraction, code: int) -> bool:
    """True when v is within a relative 2^-20 of a rounding boundary."""
    a = abs(v)
    tol = a * Fraction(1, 1 << 20)
    if code == 0:
        fl = a.numerator // a.denominator
        return abs(a - fl - Fraction(1, 2)) <= tol
    vals = [gv for gv, _ in E4M3]
    for lo, hi in zip(vals[:-1], vals[1:]):
        if lo <= a <= hi:
            return abs(a - (lo + hi) / 2) <= tol
    return False


@pytest.mark.parametrize("code", [0, 1])
def test_codes_match_exact_rational_rounding(orc, code):
    """Every finite bf16 value x in a block whose other element fixes amax:
    the code equals the exact quotient x * Q / amax rounded on the code grid
    (enumerated here from the format), except within 2^-20 of a tie where the
    fp32 reciprocal may decide."""
    Qv = Q[code]
    anchor = np.float32(3.0)
    xs = np.arange(1 << 16, dtype=np.uint32)
    xs = xs[(xs & 0x7F80) != 0x7F80].astype(np.uint16)
    block = 32
    n = xs.size
    x = np.zeros((n, block), dtype=np.uint16)
    x[:, 0] = bits([anchor])[0]
    x[:, 1] = xs
    codes, scales = orc.quantize(x, code, block)
    mism = 0
    for i in range(0, n, 7):  # every 7th value keeps the Fraction loop short
        xv = Fraction(float(f32(xs[i : i + 1])[0]))
        amax = max(abs(xv), Fraction(3))
        s = Fraction(float(scales[i, 0]))
        exact_s = amax / Qv
        # the stored scale is the fp32 value nearest amax / Q
        assert abs(s - exact_s) <= exact_s * Fraction(1, 1 << 24)
        v = xv * Qv / amax
        want = _nearest_int_even(v) & 0xFF if code == 0 else _nearest_e4m3(v)
        if int(codes[i, 1]) != want:
            assert _near_tie(v, code), (i, float(xv), int(codes[i, 1]), want)
            mism += 1
    assert mism <= 4


@pytest.mark.parametrize("code", [0, 1])
def test_reconstruction_error_bounds(orc, code):
    x = wl.activation_host(128, 1024, seed=9, outliers=("channels", 0.005, 30.0))
    codes, scales = orc.quantize(x, code, 128)
    xh = orc.dequantize(codes, scales, code, 128)
    xv = f32(x).astype(np.float64)
    hv = f32(xh).astype(np.float64)
    s = np.repeat(scales.astype(np.float64), 128, axis=1)
    err = np.abs(hv - xv)
    if code == 0:
        bound = 0.5 * s + 2.0 ** -8 * np.abs(hv) + 2.0 ** -20 * np.abs(xv)
    else:
        bound = np.maximum(2.0 ** -4 * np.abs(xv), 2.0 ** -10 * s) * (1 + 2.0 ** -20) \
            + 2.0 ** -8 * np.abs(hv)
    assert (err <= bound).all()


@pytest.mark.parametrize("code", [0, 1])
def test_zero_and_tiny_blocks(orc, code):
    x = np.zeros((3, 64), dtype=np.float32)
    x[1, 5] = 2.0 ** -65           # below 2^-64: a zero block
    x[1, 6] = -2.0 ** -66
    x[2, 7] = 2.0 ** -64           # exactly 2^-64: scaled normally
    xb = bits(x)
    codes, scales = orc.quantize(xb, code, 32)
    assert (codes[:2] == 0).all() and (scales[:2] == 0).all()
    assert scales[2, 0] == np.float32(np.float32(2.0 ** -64) / np.float32(Q[code]))
    assert codes[2, 7] == (0x7F if code == 0 else 0x7E)
    xh = orc.dequantize(codes, scales, code, 32)
    assert (xh[:2] == 0).all()


@pytest.mark.parametrize("code", [0, 1])
def test_dequantize_matches_torch_ops(orc, code):
    """xhat = bf16(value(code) * scale) against torch's fp32 multiply and cast."""
    x = wl.activation_host(64, 256, seed=3)
    codes, scales = orc.quantize(x, code, 64)
    if code == 0:
        q = torch.from_numpy(codes.view(np.int8).astype(np.float32))
    else:
        q = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float32)
    s = torch.from_numpy(scales).repeat_interleave(64, dim=1)
    ref = (q * s).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(orc.dequantize(codes, scales, code, 64), ref)


def test_row_stats(orc):
    x = np.full((2, 96), 0.75, dtype=np.float32)
    x[1] = -3.0
    xb = bits(x)
    codes, scales = orc.quantize(xb, orc.INT8, 32)
    xh = orc.dequantize(codes, scales, orc.INT8, 32)
    ss_x, ss_e = orc.row_stats(xb, xh)
    assert ss_x[0] == 96 * 0.75 ** 2 and ss_x[1] == 96 * 9.0
    assert (ss_e == 0).all()  # constant blocks sit on the grid
    r = wl.activation_host(16, 256, seed=4)
    c2, s2 = orc.quantize(r, orc.E4M3FN, 128)
    h2 = orc.dequantize(c2, s2, orc.E4M3FN, 128)
    sx, se = orc.row_stats(r, h2)
    xv, hv = f32(r).astype(np.float64), f32(h2).astype(np.float64)
    np.testing.assert_allclose(sx, np.einsum("ij,ij->i", xv, xv), rtol=1e-13)
    np.testing.assert_allclose(se, np.linalg.norm(hv - xv, axis=1) ** 2, rtol=1e-12)


def test_strided_rows(orc):
    x = wl.activation_host(8, 256, seed=6, ld=320)
    c1, s1 = orc.quantize(x, orc.INT8, 64, cols=256)
    c2, s2 = orc.quantize(np.ascontiguousarray(x[:, :256]), orc.INT8, 64)
    assert np.array_equal(c1, c2) and np.array_equal(s1, s2)
