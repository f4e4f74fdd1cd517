"""GPU parity of hilore_dequant_swiglu_bwd (backward of h = silu(g) * u with an
L operand decoded in registers) against the fp64 oracle.

The decoded operand is the oracle's dequantised bf16 value (the same bits
hilore_decompress writes); the kernel computes in fp32 and rounds each output
once to bf16, so every element must satisfy
  |gpu - truth| <= 2^-8 |truth| + 1e-5 * s,
s = |dh u| (1 + |g|) for dg and |dh g| for du: one bf16 rounding (2^-9) plus the
fp32 error of the sigmoid factor, which cancels near its zero at g ~ -1.28.
Cases: the gate or the up operand or both in L, int8 / E4M3FN at every block
size and the literal cast, strided bf16 operands, ragged row counts, the
paper-shape Qwen2.5-3B MLP activation (4096 x 11008) and its Qwen2-7B-width
counterpart (16384 x 18944) on sampled rows.
"""
import numpy as np
import pytest
import torch

from paper_2609_33570_amd import workloads as wl
from gpu_util import dev, filled, host

pytestmark = pytest.mark.gpu


def f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def check(orc, g, u, dh, got_g, got_u):
    G, U, D = (f32(a).astype(np.float64) for a in (g, u, dh))
    dg, du = orc.swiglu_bwd(G, U, D)
    for got, want, s, name in ((got_g, dg, np.abs(D * U) * (1 + np.abs(G)), "dgate"),
                               (got_u, du, np.abs(D * G), "dup")):
        gv = f32(got).astype(np.float64)
        bad = np.abs(gv - want) > 2.0 ** -8 * np.abs(want) + 1e-5 * s
        assert not bad.any(), (name, int(bad.sum()), np.argwhere(bad)[:3])


def run(hl, gate, up, code, block, dh_t, rows, cols):
    dg = filled((rows, cols), torch.bfloat16, float("nan"))
    du = filled((rows, cols), torch.bfloat16, float("nan"))
    hl.hilore_dequant_swiglu_bwd(gate, up, code, block, dh_t, dg, du)
    torch.cuda.synchronize()
    return host(dg), host(du)


@pytest.mark.parametrize("which", ["gate", "up", "both"])
@pytest.mark.parametrize("code,block", [(0, 32), (0, 128), (1, 64), (1, 128), (1, 256), (2, 0)],
                         ids=["int8-32", "int8-128", "e4m3-64", "e4m3-128", "e4m3-256", "cast"])
def test_operands_and_codes(hl, orc, which, code, block):
    rows, cols = 77, 2048 + 256
    g = wl.activation_host(rows, cols, seed=150, outliers=("channels", 0.01, 8.0))
    u = wl.activation_host(rows, cols, seed=151)
    dh = wl.normal_bf16_host(rows, cols, seed=152, sigma=0.01)
    dd = {}
    for name, x in (("gate", g), ("up", u)):
        if which in (name, "both"):
            c, s = orc.quantize(x, code, block)
            xhat = orc.dequantize(c, s, code, block)
            ct, st = dev(c), (dev(s) if s is not None else None)
            dd[name] = (hl.unit_desc(codes=ct, scales=st, rows=rows, cols=cols), xhat, (ct, st))
        else:
            xt = dev(x)
            dd[name] = (hl.unit_desc(x=xt), x, (xt,))
    got_g, got_u = run(hl, dd["gate"][0], dd["up"][0], code, block, dev(dh), rows, cols)
    check(orc, dd["gate"][1], dd["up"][1], dh, got_g, got_u)


def test_strided_bf16_and_plain(hl, orc):
    """bf16 operands with a row stride, and the all-bf16 (no L operand) case."""
    rows, cols, ld = 40, 1024, 1040
    g = wl.activation_host(rows, cols, seed=160, ld=ld)
    u = wl.activation_host(rows, cols, seed=161, ld=ld)
    dh = wl.normal_bf16_host(rows, cols, seed=162, sigma=0.01)
    gt, ut = dev(g), dev(u)
    got_g, got_u = run(hl, hl.unit_desc(x=gt, cols=cols), hl.unit_desc(x=ut, cols=cols), 1, 128,
                       dev(dh), rows, cols)
    check(orc, g[:, :cols], u[:, :cols], dh, got_g, got_u)
    c, s = orc.quantize(g, orc.E4M3FN, 128, cols=cols)
    ct, st = dev(c), dev(s)
    got_g, got_u = run(hl, hl.unit_desc(codes=ct, scales=st, rows=rows, cols=cols),
                       hl.unit_desc(x=ut, cols=cols), 1, 128, dev(dh), rows, cols)
    check(orc, orc.dequantize(c, s, orc.E4M3FN, 128), u[:, :cols], dh, got_g, got_u)


@pytest.mark.parametrize("rows,cols", [(4096, 11008), (16384, 18944)],
                         ids=["qwen2.5_3b_microbatch", "qwen2_7b_layer"])
def test_mlp_shapes(hl, orc, rows, cols):
    """The gate unit in L (E4M3FN 1x128, encoded by the library), up and dh bf16;
    checked on 64 sampled rows, the codes of those rows against the oracle."""
    g = wl.activation_device(rows, cols, 170, outliers=("channels", 0.005, 30.0))
    u = wl.activation_device(rows, cols, 171)
    dh = wl.normal_bf16_device(rows, cols, 172, 0.01)
    codes = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
    scales = torch.empty((rows, cols // 128), dtype=torch.float32, device="cuda")
    hl.hilore_compress([hl.unit_desc(x=g, codes=codes, scales=scales)], 1, 128)
    dg = torch.empty((rows, cols), dtype=torch.bfloat16, device="cuda")
    du = torch.empty((rows, cols), dtype=torch.bfloat16, device="cuda")
    hl.hilore_dequant_swiglu_bwd(hl.unit_desc(codes=codes, scales=scales, rows=rows, cols=cols),
                                 hl.unit_desc(x=u), 1, 128, dh, dg, du)
    torch.cuda.synchronize()
    sel = torch.from_numpy(np.sort(wl.rng(173, 1).choice(rows, 64, replace=False))).cuda()
    g_h = host(g[sel])
    c_h, s_h = orc.quantize(g_h, orc.E4M3FN, 128)
    assert np.array_equal(host(codes[sel]), c_h)
    check(orc, orc.dequantize(c_h, s_h, orc.E4M3FN, 128), host(u[sel]), host(dh[sel]),
          host(dg[sel]), host(du[sel]))


def test_rows_beyond_one_grid_pass(hl, orc):
    """65572 rows: the grid's row dimension stops at 65535, so the rows past it
    are taken by a second trip of the kernel's row loop (int8 1x32 gate in L,
    544 columns: one full and one partial 512-column chunk)."""
    rows, cols, block = 65535 + 37, 544, 32
    g = wl.activation_host(rows, cols, seed=170)
    u = wl.activation_host(rows, cols, seed=171)
    dh = wl.normal_bf16_host(rows, cols, seed=172, sigma=0.01)
    c, s = orc.quantize(g, 0, block)
    ct, st, ut = dev(c), dev(s), dev(u)  # descriptors hold raw pointers: keep the tensors
    got_g, got_u = run(hl, hl.unit_desc(codes=ct, scales=st, rows=rows, cols=cols),
                       hl.unit_desc(x=ut), 0, block, dev(dh), rows, cols)
    pick = np.array([0, 1, 4097, 65533, 65534, 65535, 65536, 65550, rows - 1])
    xhat = orc.dequantize(c[pick], s[pick], 0, block)
    check(orc, xhat, u[pick], dh[pick], got_g[pick], got_u[pick])
    # no row left unwritten (the outputs start as NaN)
    assert not np.isnan(f32(got_g)).any() and not np.isnan(f32(got_u)).any()
