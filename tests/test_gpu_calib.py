"""GPU parity of the calibration scalars and the update-sparsity diagnostics.

- hilore_grad_rel_err: within 1e-5 relative of the oracle's fp64 value (the
  output is fp32); exactly 0 for equal gradients and exactly 1 for g_l = 2 g_ex;
  sizes with every ragged tail, a 4096 x 4096 dW-sized pair.
- hilore_calibrate: kappa within 1e-12 relative (fp64 sums in another fixed
  order), ebar bit for bit (the same sequential sum).
- hilore_risk_score: bit for bit (the same three-factor product).
- hilore_update_sparsity: counts bit for bit; the top share within 1e-12 of the
  oracle on the same fp32 coefficients (exact selection, fp64 sums), and within
  1e-5 along the whole chain from hilore_grpo_coeffs (whose fp32 coefficients
  carry the 1e-5 tolerance).
"""
import numpy as np
import pytest
import torch

from paper_2609_33570_amd import workloads as wl
from gpu_util import assert_bytes_equal, dev, filled, host

pytestmark = pytest.mark.gpu


def rel_err_gpu(hl, a, b):
    n = a.size
    ws = torch.empty(hl.hilore_grad_rel_err_workspace_bytes(n) // 8 + 2, dtype=torch.float64,
                     device="cuda")
    y = filled(1, torch.float32, float("nan"))
    hl.hilore_grad_rel_err(dev(a) if n else filled(4, torch.float32),
                           dev(b) if n else filled(4, torch.float32), y, ws)
    torch.cuda.synchronize()
    return float(host(y)[0])


@pytest.mark.parametrize("n", [0, 1, 3, 4, 7, 4096 + 5, 1_000_003])
def test_grad_rel_err(hl, orc, n):
    rng = wl.rng(wl.BASE_SEED + 50, n)
    b = rng.standard_normal(n).astype(np.float32)
    a = (b + 1e-3 * rng.standard_normal(n)).astype(np.float32)
    got = rel_err_gpu(hl, a, b)
    want = orc.grad_rel_err(a, b)
    assert abs(got - want) <= 1e-5 * abs(want), (got, want)
    if n:
        assert rel_err_gpu(hl, b, b) == 0.0
        assert rel_err_gpu(hl, 2 * b, b) == 1.0


def test_grad_rel_err_dw_sized(hl, orc):
    """A 4096 x 4096 fp32 weight-gradient pair, the reference zero in one block
    (so eps_num matters nowhere but the sums are still exercised)."""
    g = torch.Generator(device="cuda")
    g.manual_seed(wl.BASE_SEED + 51)
    ex = torch.randn((4096, 4096), generator=g, device="cuda") * 1e-3
    ex[:64] = 0
    lo = ex + torch.randn((4096, 4096), generator=g, device="cuda") * 2e-5
    a, b = host(lo).ravel(), host(ex).ravel()
    ws = torch.empty(hl.hilore_grad_rel_err_workspace_bytes(a.size) // 8, dtype=torch.float64,
                     device="cuda")
    y = filled(1, torch.float32, float("nan"))
    hl.hilore_grad_rel_err(lo, ex, y, ws)
    torch.cuda.synchronize()
    got, want = float(host(y)[0]), orc.grad_rel_err(a, b)
    assert abs(got - want) <= 1e-5 * want, (got, want)
    # a zero reference: the eps_num floor
    hl.hilore_grad_rel_err(lo[:64], ex[:64], y, ws)
    torch.cuda.synchronize()
    want = orc.grad_rel_err(a[:64 * 4096], b[:64 * 4096])
    assert abs(float(host(y)[0]) - want) <= 1e-5 * want


def test_grad_rel_err_beyond_one_pass(hl, orc):
    """Many more 16 KiB chunks than partial slots (4 * 16384 * 1024 floats plus
    a ragged chunk and a 3-element tail: 65537 chunks over 1024 workgroups, so
    each streams 64 or 65 of them)."""
    n = 4 * 16384 * 1024 + 4096 + 3
    g = torch.Generator(device="cuda")
    g.manual_seed(wl.BASE_SEED + 52)
    ex = torch.randn(n, generator=g, device="cuda")
    lo = ex + torch.randn(n, generator=g, device="cuda") * 1e-2
    ws = torch.empty(hl.hilore_grad_rel_err_workspace_bytes(n) // 8, dtype=torch.float64,
                     device="cuda")
    assert ws.numel() == 2 * 1024
    y = filled(1, torch.float32, float("nan"))
    hl.hilore_grad_rel_err(lo, ex, y, ws)
    torch.cuda.synchronize()
    got, want = float(host(y)[0]), orc.grad_rel_err(host(lo), host(ex))
    assert abs(got - want) <= 1e-5 * want, (got, want)


def calib_case(nb, nu, nc, seed):
    rng = wl.rng(seed, 1)
    e = rng.uniform(0.1, 2.0, (nb, nu)).astype(np.float32)
    r = rng.uniform(1e-3, 5e-2, (nb, nu)).astype(np.float32)
    y = (rng.uniform(0.5, 1.5, (nb, nu)) * e * r * np.arange(1, nu + 1) % 7).astype(np.float32)
    cls = rng.integers(-1, nc + 1, nu).astype(np.int32)  # includes units of no class
    return cls, e, r, y


@pytest.mark.parametrize("nb,nu,nc", [(1, 1, 1), (8, 196, 56), (3, 300, 2), (0, 5, 3),
                                      (4, 0, 2), (16, 78, 1)])
def test_calibrate_and_risk_score(hl, orc, nb, nu, nc):
    cls, e, r, y = calib_case(nb, nu, nc, wl.BASE_SEED + 52 + nu)
    kappa = filled(max(nc, 1), torch.float64, float("nan"))
    ebar = filled(max(nu, 1), torch.float64, float("nan"))
    # empty arrays reach the library as NULL, which it accepts when their size is 0
    hl.hilore_calibrate(dev(cls), dev(e), dev(r), dev(y), nc, kappa, ebar)
    torch.cuda.synchronize()
    o_kappa, o_ebar = orc.calibrate(cls, e.reshape(nb, nu), r.reshape(nb, nu),
                                    y.reshape(nb, nu), nc)
    g_kappa = host(kappa)[:nc]
    assert np.all(np.abs(g_kappa - o_kappa) <= 1e-12 * np.abs(o_kappa)), (g_kappa, o_kappa)
    if nu == 0:
        return
    assert_bytes_equal(host(ebar)[:nu], o_ebar, "ebar")
    expo = wl.rng(wl.BASE_SEED + 53, nu).uniform(0, 3, nu).astype(np.float32)
    psi = filled(nu, torch.float64, float("nan"))
    hl.hilore_risk_score(dev(cls), dev(o_kappa) if nc else filled(1, torch.float64), dev(o_ebar),
                         dev(expo), psi)
    torch.cuda.synchronize()
    assert_bytes_equal(host(psi), orc.risk_score(cls, o_kappa, o_ebar, expo), "psi")


def sparsity_gpu(hl, coeff, flags, adv, mask, R, T, frac=0.1):
    counts = filled(3, torch.int64, -1)
    share = filled(1, torch.float64, float("nan"))
    cf = dev(coeff) if coeff.size else filled(4, torch.float32)
    fl = dev(flags) if flags.size else filled(16, torch.uint8)
    ad = dev(adv) if adv.size else filled(4, torch.float32)
    hl.hilore_update_sparsity(cf, fl, ad, dev(mask) if mask is not None else None, R, T, frac,
                              counts, share)
    torch.cuda.synchronize()
    return host(counts), float(host(share)[0])


@pytest.mark.parametrize("R,T,levels,pad", [(32, 32, 5, 0.0), (32, 1024, 1000, 0.3),
                                            (17, 61, 3, 0.5), (1, 1, 2, 0.0), (64, 1, 4, 0.2)])
@pytest.mark.parametrize("frac", [0.1, 0.01, 1.0])
def test_sparsity_exact_selection(hl, orc, R, T, levels, pad, frac):
    """Coefficients drawn from a few levels (many exact ties at the threshold)."""
    rng = wl.rng(wl.BASE_SEED + 54, R * T + levels)
    vals = (rng.standard_normal(levels) * 1e-4).astype(np.float32)
    coeff = vals[rng.integers(0, levels, R * T)]
    adv = rng.choice(np.float32([0.0, 1.0, -0.5]), R)
    flags = rng.integers(0, 4, R * T).astype(np.uint8)
    mask = (rng.random(R * T) >= pad).astype(np.uint8) if pad > 0 else None
    counts, share = sparsity_gpu(hl, coeff, flags, adv, mask, R, T, frac)
    o_counts, o_share = orc.update_sparsity(coeff.astype(np.float64), flags, adv, mask, R, T, frac)
    np.testing.assert_array_equal(counts, o_counts)
    assert abs(share - o_share) <= 1e-12 * o_share, (share, o_share)


def test_sparsity_degenerate(hl, orc):
    z = np.zeros(0, np.float32)
    counts, share = sparsity_gpu(hl, z, np.zeros(0, np.uint8), np.zeros(3, np.float32), None, 3, 0)
    assert list(counts) == [0, 0, 0] and share == 0.0
    c = np.zeros(40, np.float32)
    counts, share = sparsity_gpu(hl, c, np.zeros(40, np.uint8), np.ones(4, np.float32), None, 4, 10)
    assert list(counts) == [0, 0, 0] and share == 0.0
    c[7] = -3e-5  # one nonzero coefficient holds the whole mass
    counts, share = sparsity_gpu(hl, c, np.zeros(40, np.uint8), np.ones(4, np.float32), None, 4, 10)
    assert share == 1.0


CHAINS = [("tiny", dict(P=4, G=8, T=32)),
          ("llama3_8b_stress", dict(P=2, G=16, T=1024, pad_frac=0.3)),
          ("llama3_8b_stress_literal", dict(P=2, G=16, T=2048, pad_frac=0.3))]


@pytest.mark.parametrize("name,shape", CHAINS, ids=[c[0] for c in CHAINS])
@pytest.mark.parametrize("beta,sigma", [(0.0, 0.05), (0.0, 0.25), (1e-3, 0.25)])
def test_sparsity_after_coefficients(hl, orc, name, shape, beta, sigma):
    b = wl.grpo_batch(seed=wl.BASE_SEED + 55, with_ref=beta > 0, delta_sigma=sigma, **shape)
    R, n = b.P * b.G, b.P * b.G * b.T
    adv = filled(R, torch.float32)
    flags = filled(n, torch.uint8)
    coeff = filled(n, torch.float32)
    m = dev(b.mask) if b.mask is not None else None
    hl.hilore_grpo_coeffs(dev(b.rewards), dev(b.logp_new), dev(b.logp_old),
                          dev(b.logp_ref) if beta > 0 else None, m, b.P, b.G, b.T, 0.2, 1e-6,
                          beta, 0.0, adv, None, flags, coeff)
    counts = filled(3, torch.int64, -1)
    share = filled(1, torch.float64, float("nan"))
    hl.hilore_update_sparsity(coeff, flags, adv, m, R, b.T, 0.1, counts, share)
    torch.cuda.synchronize()
    o_adv, _, o_flags, o_coeff = orc.grpo_coeffs(b.rewards, b.logp_new, b.logp_old, b.logp_ref,
                                                 b.mask, b.P, b.G, b.T, beta=beta)
    o_counts, o_share = orc.update_sparsity(o_coeff, o_flags, o_adv, b.mask, R, b.T, 0.1)
    np.testing.assert_array_equal(host(counts), o_counts)
    got = float(host(share)[0])
    assert abs(got - o_share) <= 1e-5 * o_share, (got, o_share)


def test_deterministic(hl, orc):
    """Fixed-order fp64 sums: repeated calls agree bit for bit (the relative
    error at two sizes with ragged tails, the sparsity counts and share on the
    path that does not keep the magnitudes in LDS)."""
    rng = wl.rng(wl.BASE_SEED + 56, 1)
    for n in (3_000_001, 65_541):
        b = rng.standard_normal(n).astype(np.float32)
        a = (b + 1e-2 * rng.standard_normal(n)).astype(np.float32)
        assert rel_err_gpu(hl, a, b) == rel_err_gpu(hl, a, b)
    R, T = 64, 1024  # 65536 slots: past the LDS cache, every pass reads memory
    coeff = (rng.standard_normal(R * T) * 1e-4).astype(np.float32)
    flags = rng.integers(0, 4, R * T).astype(np.uint8)
    adv = rng.standard_normal(R).astype(np.float32)
    c1, s1 = sparsity_gpu(hl, coeff, flags, adv, None, R, T)
    c2, s2 = sparsity_gpu(hl, coeff, flags, adv, None, R, T)
    assert np.array_equal(c1, c2) and s1 == s2
    _, o_share = orc.update_sparsity(coeff.astype(np.float64), flags, adv, None, R, T, 0.1)
    assert abs(s1 - o_share) <= 1e-12 * o_share
