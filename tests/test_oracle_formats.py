"""Pins of the oracle's number formats against torch's own casts.

bf16 round-to-nearest-even and OCP E4M3FN round-to-nearest-even are the two
roundings the codec of App. B.1 (Eq. fp8-roundtrip) is built from.  torch's
CPU casts are an independent implementation of the same rules, so the oracle
must agree with them on every value tried (E4M3FN only where torch's cast does
not overflow: |v| < 464; torch's cast turns larger values into NaN, while the
codec here saturates and never produces such values).
"""
import numpy as np
import pytest
import torch


def _f32(bits):
    return np.asarray(bits, dtype=np.uint32).view(np.float32)


def _torch_bf16_bits(v):
    return torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _torch_e4m3_bits(v):
    return torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_bf16_rne_matches_torch_structured(orc):
    hi = np.arange(1 << 16, dtype=np.uint32)
    hi = hi[(hi & 0x7F80) != 0x7F80]  # finite
    lows = np.array([0x0000, 0x0001, 0x4000, 0x7FFF, 0x8000, 0x8001, 0xC000, 0xFFFF],
                    dtype=np.uint32)
    bits = (hi[:, None] << 16 | lows[None, :]).ravel()
    v = _f32(bits)
    assert np.array_equal(orc.bf16_rne(v), _torch_bf16_bits(v))


def test_bf16_rne_matches_torch_random(orc):
    g = np.random.default_rng(11)
    bits = g.integers(0, 1 << 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    bits = bits[(bits & 0x7F800000) != 0x7F800000]
    v = _f32(bits)
    assert np.array_equal(orc.bf16_rne(v), _torch_bf16_bits(v))


def test_bf16_rne_ties_and_overflow(orc):
    # 1 + 2^-8 is the midpoint of 1 and 1 + 2^-7: ties go to the even mantissa (1.0)
    assert orc.bf16_rne(np.float32([1.00390625]))[0] == 0x3F80
    # 1 + 3 * 2^-8 is the midpoint of 1 + 2^-7 and 1 + 2^-6: even is 1 + 2^-6
    assert orc.bf16_rne(np.float32([1.01171875]))[0] == 0x3F82
    # largest finite fp32 rounds past the largest bf16 -> +inf
    assert orc.bf16_rne(np.float32([3.4028235e38]))[0] == 0x7F80


def _e4m3_values():
    """All finite non-negative E4M3FN values by the format definition."""
    vals = []
    for e in range(16):
        for m in range(8):
            if e == 15 and m == 7:
                continue
            vals.append(m * 2.0 ** -9 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7))
    return np.array(vals)


def test_e4m3_decode_matches_torch(orc):
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float32).numpy()
    mine = np.array([orc.e4m3fn_decode(int(c)) for c in codes])
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(mine))
    assert nan.sum() == 2 and nan[0x7F] and nan[0xFF]
    assert np.array_equal(ref[~nan].astype(np.float64), mine[~nan])


def test_e4m3_rne_matches_torch(orc):
    g = np.random.default_rng(12)
    parts = []
    # every bf16-grid magnitude below 464, with low halves around the tie points
    hi = np.arange(0, 0x43E8, dtype=np.uint32)
    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    parts.append(_f32((hi[:, None] << 16 | lows[None, :]).ravel()))
    # exact midpoints between neighbouring E4M3FN values, and one ulp either side
    ev = _e4m3_values()
    mid = ((ev[:-1] + ev[1:]) / 2).astype(np.float32)
    parts += [mid, np.nextafter(mid, np.float32(0)), np.nextafter(mid, np.float32(1e9))]
    parts.append(np.float32([448.0, 448.5, 460.0, 463.99997]))
    parts.append(g.uniform(-448, 448, 1 << 20).astype(np.float32))
    parts.append((np.exp2(g.uniform(-14, 8.8, 1 << 20)) * 0.999).astype(np.float32))
    v = np.concatenate(parts).astype(np.float32)
    v = np.concatenate([v, -v])
    v = v[np.abs(v) < 464]
    assert np.array_equal(orc.e4m3fn_rne(v), _torch_e4m3_bits(v))


def test_e4m3_sign_of_zero_and_saturation(orc):
    out = orc.e4m3fn_rne(np.float32([0.0, -0.0, -1e-30, 1e-30, 470.0, -1000.0, 448.00003]))
    assert list(out) == [0x00, 0x80, 0x80, 0x00, 0x7E, 0xFE, 0x7E]


def test_code_values(orc):
    assert orc.code_value(orc.INT8, 0x81) == -127.0
    assert orc.code_value(orc.INT8, 0x7F) == 127.0
    assert orc.code_value(orc.E4M3FN, 0x7E) == 448.0
    assert orc.code_value(orc.E4M3FN, 0x01) == 2.0 ** -9
    assert orc.code_value(orc.E4M3FN, 0x08) == 2.0 ** -6


# --- the paper's literal codec: a plain torch.float8_e4m3fn cast (App. B.1,
# Eq. fp8-roundtrip, "without scales, zero-points, or outlier tensors") -------

def test_e4m3_cast_matches_torch_on_every_bf16(orc):
    """The cast of every bf16 bit pattern (finite, infinite and NaN) equals
    torch's own CPU cast byte for byte, overflow-to-NaN included."""
    bits = (np.arange(1 << 16, dtype=np.uint32) << 16)
    v = _f32(bits)
    ref = torch.from_numpy(bits.astype(np.uint32).view(np.int32) >> 16).to(torch.int16)
    ref = ref.view(torch.bfloat16).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(orc.e4m3fn_cast(v), ref)


def test_e4m3_cast_matches_torch_random_fp32(orc):
    g = np.random.default_rng(12)
    bits = g.integers(0, 1 << 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    # concentrate half of the samples on the E4M3FN range and its overflow edge
    mags = g.uniform(0, 520, size=1 << 19).astype(np.float32) * np.where(g.random(1 << 19) < .5, -1, 1)
    v = np.concatenate([_f32(bits), mags.astype(np.float32)])
    assert np.array_equal(orc.e4m3fn_cast(v), _torch_e4m3_bits(v))


def test_e4m3_cast_overflow_edge(orc):
    # 464 is the midpoint of 448 and the would-be 480: ties to even -> 448;
    # anything past it has no encoding -> NaN with the sign kept
    v = np.float32([448.0, 463.99997, 464.0, np.nextafter(np.float32(464), np.float32(1e9)),
                    -464.0, -465.0, np.inf, -np.inf, -0.0])
    assert orc.e4m3fn_cast(v).tolist() == [0x7E, 0x7E, 0x7E, 0x7F, 0xFE, 0xFF, 0x7F, 0xFF, 0x80]


def test_e4m3_cast_back_matches_torch(orc):
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).to(torch.bfloat16).view(torch.int16).numpy()
    ref = ref.view(np.uint16)
    ours = np.array([orc.e4m3fn_cast_to_bf16(c) for c in range(256)], dtype=np.uint16)
    assert np.array_equal(ours, ref)
    assert ours[0x7F] == ours[0xFF] == 0x7FC0


def test_literal_codec_roundtrip_is_torch_roundtrip(orc):
    """quantize/dequantize with the literal code reproduce
    x.to(float8_e4m3fn).to(bfloat16) of torch on a tensor with overflow."""
    g = np.random.default_rng(13)
    x = (g.standard_normal((37, 96)) * 120).astype(np.float32)
    x[3, 5] = 600.0
    x[7, 9] = -1e30
    xb = torch.from_numpy(x).to(torch.bfloat16)
    xu = xb.view(torch.int16).numpy().view(np.uint16)
    codes, scales = orc.quantize(xu, orc.E4M3FN_CAST, 0)
    assert scales is None
    ref_c = xb.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes, ref_c)
    xh = orc.dequantize(codes, None, orc.E4M3FN_CAST, 0)
    ref_h = xb.to(torch.float8_e4m3fn).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(xh, ref_h)
    assert xh[3, 5] == 0x7FC0 and xh[7, 9] == 0x7FC0
