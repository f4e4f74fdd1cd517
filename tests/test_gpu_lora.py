"""GPU parity of hilore_dequant_lora_grad (the LoRA adapter gradient on an L
unit) against the oracle.

  - integer-valued operands: every partial sum is an integer below 2^24, so
    fp32 accumulation is exact in any order and the result (times a power-of-
    two scale) must equal the oracle bit for bit;
  - general operands: relative Frobenius error against the fp64 oracle on the
    same bf16 operand (variant 1, only fp32 accumulation differs: <= 1e-5) and
    on the unrounded dequantisation (variant 0: <= 2e-2), for every code and
    block size;
  - ragged K, M and even adapter ranks 2..98 (one-block passes and cooperative
    passes of up to 80 rows, dh read in 16-byte chunks or in pairs),
    accumulation, K = 0, and the Qwen2-7B-width MLP and hidden units (16384 x
    18944 and 16384 x 3584, fp8 1x128, rank 16, and rank 80 on the hidden
    unit) on sampled columns.
"""
import numpy as np
import pytest
import torch

from paper_2609_33570_amd import workloads as wl
from gpu_util import assert_bytes_equal, dev, filled, host, rel_fro

pytestmark = pytest.mark.gpu


def gpu_lora(hl, codes, scales, code, block, dh, scale=2.0, accumulate=False, da0=None):
    K, M = codes.shape
    r = dh.shape[1]
    da = dev(da0.astype(np.float32)) if da0 is not None else filled((r, M), torch.float32,
                                                                   float("nan"))
    ws = torch.empty(hl.hilore_lora_grad_workspace_bytes(K, M, r) // 4, dtype=torch.float32,
                     device="cuda")
    sc = None if scales is None else (dev(scales) if K else filled((1, M // block), torch.float32))
    hl.hilore_dequant_lora_grad(dev(codes) if K else filled((1, M), torch.uint8), sc, code, block,
                                dev(dh) if K else filled((1, r), torch.bfloat16), da, K, M, r,
                                scale, accumulate, ws)
    torch.cuda.synchronize()
    return host(da)


@pytest.mark.parametrize("r", [16, 42, 48, 80, 96])
def test_integer_exact(hl, orc, r):
    """Ranks above 16 run the cooperative kernel (passes of up to 80 rows: 96 is
    80 + 16); 42 is not a multiple of 8, so its dh block is read in pairs."""
    g = np.random.default_rng(7 + r)
    K, M = 16384, 512
    q = g.integers(-7, 8, size=(K, M)) * 16
    codes = q.astype(np.int8).view(np.uint8)
    scales = np.full((K, M // 128), 1 / 16, dtype=np.float32)
    dh = wl.to_bf16_bits(g.integers(-8, 9, size=(K, r)).astype(np.float32))
    got = gpu_lora(hl, codes, scales, 0, 128, dh, scale=2.0)
    want = orc.lora_down_grad(codes, scales, 0, 128, dh, scale=2.0, variant=1)
    assert_bytes_equal(got, want.astype(np.float32), "dA")


@pytest.mark.parametrize("code", [0, 1], ids=["int8", "e4m3fn"])
@pytest.mark.parametrize("block", [32, 64, 128, 256])
def test_codes_and_blocks(hl, orc, code, block):
    K, M, r = 1000, 768, 16
    x = wl.activation_host(K, M, seed=70 + block, outliers=("channels", 0.005, 30.0))
    codes, scales = orc.quantize(x, code, block)
    dh = wl.normal_bf16_host(K, r, seed=80 + block, sigma=0.05)
    got = gpu_lora(hl, codes, scales, code, block, dh)
    v1 = orc.lora_down_grad(codes, scales, code, block, dh, scale=2.0, variant=1)
    v0 = orc.lora_down_grad(codes, scales, code, block, dh, scale=2.0, variant=0)
    assert rel_fro(got, v1) <= 1e-5
    assert rel_fro(got, v0) <= 2e-2


def test_literal_cast(hl, orc):
    K, M, r = 700, 512, 16
    x = wl.activation_host(K, M, seed=90)
    codes, _ = orc.quantize(x, orc.E4M3FN_CAST, 0)
    dh = wl.normal_bf16_host(K, r, seed=91, sigma=0.05)
    got = gpu_lora(hl, codes, None, orc.E4M3FN_CAST, 0, dh, scale=1.0)
    want = orc.lora_down_grad(codes, None, orc.E4M3FN_CAST, 0, dh, scale=1.0, variant=1)
    assert rel_fro(got, want) <= 1e-5


@pytest.mark.parametrize("K,M,r", [(1, 16, 16), (31, 272, 2), (33, 256, 8), (64, 4112, 18),
                                   (517, 1040, 40), (2048, 256, 16), (95, 48, 32), (47, 528, 6),
                                   (300, 528, 66), (1000, 256, 80), (65, 784, 98)])
def test_ragged_shapes(hl, orc, K, M, r):
    """Widths that are multiples of 32 use E4M3FN with 32-wide blocks; the others
    (multiples of 16 only) use the literal cast, which has no blocks."""
    x = wl.activation_host(K, M, seed=100 + K, outliers=("entries", 0.01, 20.0))
    code, block = (orc.E4M3FN, 32) if M % 32 == 0 else (orc.E4M3FN_CAST, 0)
    codes, scales = orc.quantize(x, code, block)
    dh = wl.normal_bf16_host(K, r, seed=110 + r, sigma=0.05)
    got = gpu_lora(hl, codes, scales, code, block, dh)
    v1 = orc.lora_down_grad(codes, scales, code, block, dh, scale=2.0, variant=1)
    assert rel_fro(got, v1) <= 1e-5


@pytest.mark.parametrize("r", [16, 48])
def test_accumulate_and_empty(hl, orc, r):
    K, M = 300, 512
    x = wl.activation_host(K, M, seed=120)
    codes, scales = orc.quantize(x, orc.INT8, 64)
    dh = wl.normal_bf16_host(K, r, seed=121, sigma=0.05)
    da0 = wl.rng(122, 1).standard_normal((r, M)).astype(np.float32)
    got = gpu_lora(hl, codes, scales, orc.INT8, 64, dh, accumulate=True, da0=da0)
    want = da0 + orc.lora_down_grad(codes, scales, orc.INT8, 64, dh, scale=2.0, variant=1)
    assert rel_fro(got, want) <= 1e-6
    empty_c = np.zeros((0, M), np.uint8)
    empty_s = np.zeros((0, M // 64), np.float32)
    empty_h = np.zeros((0, r), np.uint16)
    assert not np.any(gpu_lora(hl, empty_c, empty_s, orc.INT8, 64, empty_h))
    np.testing.assert_array_equal(
        gpu_lora(hl, empty_c, empty_s, orc.INT8, 64, empty_h, accumulate=True, da0=da0), da0)


def test_narrow_unit_accumulate(hl, orc):
    """A narrow unit (7 strips, 131 k-steps: each strip split into parts of
    unequal length, one workgroup each) with two 16-row passes, accumulating."""
    K, M, r = 4096 + 96, 1792, 18
    x = wl.activation_host(K, M, seed=125, outliers=("channels", 0.005, 30.0))
    codes, scales = orc.quantize(x, orc.INT8, 64)
    dh = wl.normal_bf16_host(K, r, seed=126, sigma=0.05)
    da0 = wl.rng(127, 1).standard_normal((r, M)).astype(np.float32)
    got = gpu_lora(hl, codes, scales, orc.INT8, 64, dh, accumulate=True, da0=da0)
    want = da0 + orc.lora_down_grad(codes, scales, orc.INT8, 64, dh, scale=2.0, variant=1)
    assert rel_fro(got, want) <= 1e-6


def test_deterministic(hl, orc):
    K, M, r = 4096, 2048, 16
    x = wl.activation_host(K, M, seed=130)
    codes, scales = orc.quantize(x, orc.E4M3FN, 128)
    dh = wl.normal_bf16_host(K, r, seed=131, sigma=0.05)
    a = gpu_lora(hl, codes, scales, orc.E4M3FN, 128, dh)
    b = gpu_lora(hl, codes, scales, orc.E4M3FN, 128, dh)
    assert_bytes_equal(a, b, "repeat")


@pytest.mark.parametrize("M,unit,r", [(18944, 1, 16), (3584, 0, 16), (3584, 0, 80)],
                         ids=["mlp_18944", "hidden_3584", "hidden_3584_qkvgu"])
def test_qwen2_7b_units(hl, orc, M, unit, r):
    """The Qwen2-7B-width units at full size (16384 x 18944 MLP: 74 strips, the
    stream-K plan; 16384 x 3584 hidden: 14 strips, one workgroup per strip
    part), fp8 1x128, one rank-16 adapter, and on the hidden unit the five
    rank-16 adapters that share it (q, k, v, gate, up: r = 80, one pass): the
    first 2048 columns (8 strips) and 24 columns drawn from the rest, against
    the oracle on codes the oracle recomputes."""
    w = wl.QWEN2_7B_LAYER
    K, block, code = 16384, 128, hl.HILORE_CODE_FP8_E4M3FN
    x = wl.activation_device(K, M, w.seed * 10 + unit, outliers=w.outliers)
    codes = torch.empty((K, M), dtype=torch.uint8, device="cuda")
    scales = torch.empty((K, M // block), dtype=torch.float32, device="cuda")
    hl.hilore_compress([hl.unit_desc(x=x, codes=codes, scales=scales)], code, block)
    dh = wl.normal_bf16_device(K, r, 140, 0.05)
    da = filled((r, M), torch.float32, float("nan"))
    ws = torch.empty(hl.hilore_lora_grad_workspace_bytes(K, M, r) // 4, dtype=torch.float32,
                     device="cuda")
    hl.hilore_dequant_lora_grad(codes, scales, code, block, dh, da, K, M, r, 2.0, False, ws)
    torch.cuda.synchronize()
    got = host(da)
    x_h = host(x)
    del x
    dh_h = host(dh)
    # the codes are the library's; check them against the oracle on the columns used
    cols = np.unique(np.concatenate([np.arange(0, 2048),
                                     wl.rng(141, 1).choice(M, 24, replace=False)]))
    blocks = np.unique(cols // block)
    sub_cols = (blocks[:, None] * block + np.arange(block)[None, :]).ravel()
    o_codes, o_scales = orc.quantize(np.ascontiguousarray(x_h[:, sub_cols]), code, block)
    assert_bytes_equal(host(codes)[:, sub_cols], o_codes, "codes")
    want = orc.lora_down_grad(o_codes, o_scales, code, block, dh_h, scale=2.0, variant=1)
    pos = {c: i for i, c in enumerate(sub_cols)}
    idx = np.array([pos[c] for c in cols])
    assert rel_fro(got[:, cols], want[:, idx]) <= 1e-5
    v0 = orc.lora_down_grad(o_codes, o_scales, code, block, dh_h, scale=2.0, variant=0)
    assert rel_fro(got[:, cols], v0[:, idx]) <= 2e-2
