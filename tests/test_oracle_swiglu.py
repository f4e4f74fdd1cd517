"""Pins of the oracle's gated-MLP activation backward (h = silu(g) * u, the
MLP of the evaluated Qwen/Llama models whose gate and up activations can be L
units): fp64 PyTorch autograd of the forward, central finite differences, and
the closed forms at g = 0 and for large |g|."""
import numpy as np
import pytest
import torch


def test_against_autograd(orc):
    g0 = np.random.default_rng(1)
    n = 5000
    g = g0.standard_normal(n) * 3
    u = g0.standard_normal(n)
    dh = g0.standard_normal(n) * 1e-2
    gt = torch.tensor(g, requires_grad=True)
    ut = torch.tensor(u, requires_grad=True)
    (torch.nn.functional.silu(gt) * ut).backward(torch.tensor(dh))
    dg, du = orc.swiglu_bwd(g, u, dh)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-12, atol=1e-18)
    np.testing.assert_allclose(du, ut.grad.numpy(), rtol=1e-12, atol=1e-18)


def test_finite_differences(orc):
    g0 = np.random.default_rng(2)
    g = g0.standard_normal(200) * 4
    u = g0.standard_normal(200)
    dh = np.ones(200)
    f = lambda gg, uu: gg / (1 + np.exp(-gg)) * uu  # noqa: E731
    h = 1e-6
    dg, du = orc.swiglu_bwd(g, u, dh)
    np.testing.assert_allclose(dg, (f(g + h, u) - f(g - h, u)) / (2 * h), rtol=1e-6, atol=1e-9)
    np.testing.assert_allclose(du, (f(g, u + h) - f(g, u - h)) / (2 * h), rtol=1e-6, atol=1e-9)


def test_closed_forms(orc):
    u = np.array([2.0, -3.0, 0.5])
    dh = np.array([1.0, 0.25, -4.0])
    dg, du = orc.swiglu_bwd(np.zeros(3), u, dh)
    np.testing.assert_array_equal(du, np.zeros(3))        # silu(0) = 0
    np.testing.assert_array_equal(dg, 0.5 * dh * u)       # silu'(0) = 1/2
    dg, du = orc.swiglu_bwd(np.full(3, 60.0), u, dh)      # sigmoid -> 1: silu(g) -> g
    np.testing.assert_allclose(du, 60.0 * dh, rtol=1e-15)
    np.testing.assert_allclose(dg, dh * u, rtol=1e-15)
    dg, du = orc.swiglu_bwd(np.full(3, -60.0), u, dh)     # sigmoid -> 0
    assert np.all(np.abs(du) < 1e-23) and np.all(np.abs(dg) < 1e-21)
