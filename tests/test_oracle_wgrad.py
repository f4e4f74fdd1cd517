"""Pins of the oracle's weight gradient on reconstructed activations,
dW = deq(X)^T dY (the full-parameter wgrad of App. D; compared by the
relative Frobenius error of Eq. measured-gradient-error).

Pinned against exact integer arithmetic (numpy int64 matmul), numpy's fp64
matmul on the dequantised operand, one-hot columns (column sums), and the
bf16-rounding bound between the two dequantisation variants.
"""
import numpy as np
import pytest

from paper_2609_33570_amd import workloads as wl


def f32(bf):
    return (np.asarray(bf, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def test_integer_exact(orc):
    g = np.random.default_rng(1)
    K, M, N = 70, 64, 48
    q = g.integers(-7, 8, size=(K, M)) * 16          # int8 codes, multiples of 16
    codes = q.astype(np.int8).view(np.uint8)
    scales = np.full((K, M // 32), 1 / 16, dtype=np.float32)
    dyi = g.integers(-8, 9, size=(K, N))
    dy = wl.to_bf16_bits(dyi.astype(np.float32))
    want = (q // 16).T @ dyi
    for variant in (0, 1):
        dw = orc.wgrad(codes, scales, orc.INT8, 32, dy, variant=variant)
        assert np.array_equal(dw, want.astype(np.float64))


@pytest.mark.parametrize("code", [0, 1])
def test_matches_numpy_on_dequantised_operand(orc, code):
    K, M, N = 96, 128, 80
    x = wl.activation_host(K, M, seed=31, outliers=("channels", 0.02, 30.0))
    codes, scales = orc.quantize(x, code, 64)
    xh = f32(orc.dequantize(codes, scales, code, 64)).astype(np.float64)
    dy = wl.normal_bf16_host(K, N, seed=32, sigma=0.02)
    ref = xh.T @ f32(dy).astype(np.float64)
    dw1 = orc.wgrad(codes, scales, code, 64, dy, variant=1)
    np.testing.assert_allclose(dw1, ref, rtol=1e-12, atol=1e-14 * np.abs(ref).max())
    dw0 = orc.wgrad(codes, scales, code, 64, dy, variant=0)
    rel = np.linalg.norm(dw0 - dw1) / np.linalg.norm(dw0)
    assert rel < 2.0 ** -8
    # subtiles and single entries agree with the full result
    sub = orc.wgrad(codes, scales, code, 64, dy, 32, 96, 8, 40, variant=1)
    assert np.array_equal(sub, dw1[32:96, 8:40])
    ii = np.array([0, 5, 127, 64])
    jj = np.array([79, 0, 3, 40])
    ent = orc.wgrad_entries(codes, scales, code, 64, dy, ii, jj, variant=1)
    np.testing.assert_allclose(ent, dw1[ii, jj], rtol=1e-14)


def test_ones_column_gives_column_sums(orc):
    K, M, N = 50, 64, 16
    x = wl.activation_host(K, M, seed=33)
    codes, scales = orc.quantize(x, orc.E4M3FN, 32)
    dyv = np.zeros((K, N), dtype=np.float32)
    dyv[:, 3] = 1.0
    dy = wl.to_bf16_bits(dyv)
    dw = orc.wgrad(codes, scales, orc.E4M3FN, 32, dy, variant=1)
    xh = f32(orc.dequantize(codes, scales, orc.E4M3FN, 32)).astype(np.float64)
    np.testing.assert_allclose(dw[:, 3], xh.sum(axis=0), rtol=1e-14)
    assert (dw[:, np.arange(N) != 3] == 0).all()


def test_literal_cast_code_matches_torch_cast_operand(orc):
    """With the literal codec the operand is torch's own bf16 -> float8_e4m3fn
    -> bf16 round trip; the oracle's wgrad equals numpy on it."""
    import torch
    K, M, N = 80, 64, 40
    x = wl.activation_host(K, M, seed=34, outliers=("channels", 0.05, 30.0))
    xt = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16)
    xh = xt.to(torch.float8_e4m3fn).to(torch.float32).numpy().astype(np.float64)
    codes, scales = orc.quantize(x, orc.E4M3FN_CAST, 0)
    dy = wl.normal_bf16_host(K, N, seed=35, sigma=0.02)
    ref = xh.T @ f32(dy).astype(np.float64)
    for variant in (0, 1):
        dw = orc.wgrad(codes, None, orc.E4M3FN_CAST, 0, dy, variant=variant)
        np.testing.assert_allclose(dw, ref, rtol=1e-12, atol=1e-14 * np.abs(ref).max())
