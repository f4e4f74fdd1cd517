"""GPU parity of hilore_dequant_wgrad against the oracle.

  - integer-valued operands: every partial sum is an integer below 2^24, so
    fp32 accumulation is exact in any order and the result must equal the
    oracle bit for bit;
  - general operands: relative Frobenius error (Eq. measured-gradient-error)
    against the fp64 oracle on the same bf16 operand (variant 1, only fp32
    accumulation differs: <= 1e-5) and on the unrounded dequantisation
    (variant 0: <= 2e-2);
  - ragged M, N and K, accumulation into an existing dW, K = 0.
"""
import numpy as np
import pytest
import torch

from paper_2609_33570_amd import workloads as wl
from gpu_util import assert_bytes_equal, dev, filled, host, rel_fro

pytestmark = pytest.mark.gpu


def gpu_wgrad(hl, codes, scales, code, block, dy, accumulate=False, dw0=None):
    K, M = codes.shape
    N = dy.shape[1]
    dw = dev(dw0.astype(np.float32)) if dw0 is not None else filled((M, N), torch.float32,
                                                                   float("nan"))
    hl.hilore_dequant_wgrad(dev(codes) if K else filled((1, M), torch.uint8),
                            dev(scales) if K else filled((1, M // block), torch.float32),
                            code, block, dev(dy) if K else filled((1, N), torch.bfloat16),
                            dw, K, M, N, accumulate)
    torch.cuda.synchronize()
    return host(dw)


def test_integer_exact(hl, orc):
    g = np.random.default_rng(5)
    K, M, N = 16384, 512, 512
    q = g.integers(-7, 8, size=(K, M)) * 16
    codes = q.astype(np.int8).view(np.uint8)
    scales = np.full((K, M // 128), 1 / 16, dtype=np.float32)
    dy = wl.to_bf16_bits(g.integers(-8, 9, size=(K, N)).astype(np.float32))
    got = gpu_wgrad(hl, codes, scales, 0, 128, dy)
    want = orc.wgrad(codes, scales, 0, 128, dy, variant=1)
    assert_bytes_equal(got, want.astype(np.float32), "dW")


@pytest.mark.parametrize("code", [0, 1], ids=["int8", "e4m3fn"])
@pytest.mark.parametrize("block", [32, 64, 128, 256])
def test_ragged_shapes(hl, orc, code, block):
    K, M, N = 1000, 768, 264 + 8
    x = wl.activation_host(K, M, seed=50 + block, outliers=("channels", 0.005, 30.0))
    codes, scales = orc.quantize(x, code, block)
    dy = wl.normal_bf16_host(K, N, seed=60 + block, sigma=0.02)
    got = gpu_wgrad(hl, codes, scales, code, block, dy)
    v1 = orc.wgrad(codes, scales, code, block, dy, variant=1)
    v0 = orc.wgrad(codes, scales, code, block, dy, variant=0)
    assert rel_fro(got, v1) <= 1e-5
    assert rel_fro(got, v0) <= 2e-2


@pytest.mark.parametrize("K,M,N", [(1, 256, 256), (63, 128, 8), (65, 256, 264), (200, 544, 520),
                                   (64, 2048, 256)])
def test_small_and_edge_tiles(hl, orc, K, M, N):
    x = wl.activation_host(K, M, seed=K + M + N)
    codes, scales = orc.quantize(x, 1, 32)
    dy = wl.normal_bf16_host(K, N, seed=K * N, sigma=1.0)
    got = gpu_wgrad(hl, codes, scales, 1, 32, dy)
    assert rel_fro(got, orc.wgrad(codes, scales, 1, 32, dy, variant=1)) <= 1e-5


def test_accumulate(hl, orc):
    K, M, N = 300, 512, 256
    x = wl.activation_host(K, M, seed=71)
    codes, scales = orc.quantize(x, 0, 64)
    dy = wl.normal_bf16_host(K, N, seed=72, sigma=0.5)
    dw0 = np.random.default_rng(73).normal(size=(M, N)).astype(np.float32)
    got = gpu_wgrad(hl, codes, scales, 0, 64, dy, accumulate=True, dw0=dw0)
    want = dw0.astype(np.float64) + orc.wgrad(codes, scales, 0, 64, dy, variant=1)
    assert rel_fro(got, want) <= 1e-6


def test_empty_contraction(hl, orc):
    M, N = 256, 512
    got = gpu_wgrad(hl, np.zeros((0, M), np.uint8), np.zeros((0, M // 128), np.float32), 1, 128,
                    np.zeros((0, N), np.uint16))
    assert (got == 0).all()
    dw0 = np.ones((M, N), np.float32)
    got = gpu_wgrad(hl, np.zeros((0, M), np.uint8), np.zeros((0, M // 128), np.float32), 1, 128,
                    np.zeros((0, N), np.uint16), accumulate=True, dw0=dw0)
    assert (got == 1).all()


def test_deterministic(hl, orc):
    K, M, N = 2048, 1024, 1024
    x = wl.activation_host(K, M, seed=81)
    codes, scales = orc.quantize(x, 1, 128)
    dy = wl.normal_bf16_host(K, N, seed=82, sigma=0.02)
    a = gpu_wgrad(hl, codes, scales, 1, 128, dy)
    b = gpu_wgrad(hl, codes, scales, 1, 128, dy)
    assert_bytes_equal(a, b, "repeat")


def test_literal_cast_integer_exact(hl, orc):
    """Literal cast codes (no scales) of small integers: exact in any order."""
    g = np.random.default_rng(15)
    K, M, N = 4096, 256, 264
    xi = g.integers(-8, 9, size=(K, M)).astype(np.float32)
    codes, _ = orc.quantize(wl.to_bf16_bits(xi), 2, 0)
    dy = wl.to_bf16_bits(g.integers(-8, 9, size=(K, N)).astype(np.float32))
    dw = filled((M, N), torch.float32, float("nan"))
    hl.hilore_dequant_wgrad(dev(codes), None, 2, 0, dev(dy), dw, K, M, N, False)
    torch.cuda.synchronize()
    want = orc.wgrad(codes, None, 2, 0, dy, variant=1)
    assert_bytes_equal(host(dw), want.astype(np.float32), "dW")


def test_literal_cast_activations(hl, orc):
    K, M, N = 1000, 512, 264
    x = wl.activation_host(K, M, seed=16, outliers=("channels", 0.01, 30.0))
    codes, _ = orc.quantize(x, 2, 0)
    assert not ((codes & 0x7F) == 0x7F).any()
    dy = wl.normal_bf16_host(K, N, seed=17, sigma=0.02)
    dw = filled((M, N), torch.float32, float("nan"))
    hl.hilore_dequant_wgrad(dev(codes), None, 2, 0, dev(dy), dw, K, M, N, False)
    torch.cuda.synchronize()
    assert rel_fro(host(dw), orc.wgrad(codes, None, 2, 0, dy, variant=1)) <= 1e-5
