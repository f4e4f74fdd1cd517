"""Pin of the LoRA adapter gradient read off the oracle's weight gradient
(the full-parameter form X^T dY, already pinned by integer and numpy checks).

Independent reference: fp64 autograd (PyTorch on the CPU) of the LoRA layer
forward y = X W^T + (alpha / r) (X A^T) B^T with the paper's adapter settings
(rank 16, alpha 32, App. D.1.1), X the dequantised L unit.  The gradient of A
for an arbitrary upstream gradient G must equal the oracle's dA computed from
dh = G B alone, which pins both the reading dA = s (G B)^T X and the transpose.
"""
import numpy as np
import torch

from paper_2609_33570_amd import workloads as wl


def test_lora_grad_equals_autograd(orc):
    K, M, out, r, alpha = 96, 256, 48, 16, 32.0
    x = wl.activation_host(K, M, seed=61, outliers=("channels", 0.02, 30.0))
    codes, scales = orc.quantize(x, orc.E4M3FN, 128)
    xhat = orc.bf16_to_f32(orc.dequantize(codes, scales, orc.E4M3FN, 128)).astype(np.float64)
    g = wl.rng(62, 1)
    W = torch.tensor(g.standard_normal((out, M)), dtype=torch.float64)
    A = torch.tensor(g.standard_normal((r, M)) * 0.02, dtype=torch.float64, requires_grad=True)
    B = torch.tensor(g.standard_normal((out, r)) * 0.02, dtype=torch.float64)
    G = torch.tensor(g.standard_normal((K, out)), dtype=torch.float64)
    X = torch.tensor(xhat)
    y = X @ W.T + (alpha / r) * (X @ A.T) @ B.T
    y.backward(G)
    dh = (G @ B).numpy()
    # the oracle takes dh as bf16: use values exact in bf16 by rounding dh first
    dh16 = orc.bf16_rne(dh.astype(np.float32)).reshape(K, r)
    dh_exact = orc.bf16_to_f32(dh16).astype(np.float64)
    want = (alpha / r) * dh_exact.T @ xhat
    got = orc.lora_down_grad(codes, scales, orc.E4M3FN, 128, dh16, scale=alpha / r, variant=1)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)
    # and autograd's dA differs from it only by the bf16 rounding of dh
    rel = np.linalg.norm(got - A.grad.numpy()) / np.linalg.norm(A.grad.numpy())
    assert rel < 1e-2
