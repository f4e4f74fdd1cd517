"""Pins of the oracle's calibration scalars and update diagnostics.

- y (App. B.1 Eq. app-calibration-error; Sec. 3.4 Eq. calibration-metrics):
  zero for identical gradients, exactly 1 for g_l = 2 g_ex, the eps_num floor
  for a zero reference, invariance under a common power-of-two scaling, and
  numpy's fp64 norms.
- kappa (Eqs. app-kappa / susceptibility): the one-column non-negative least
  squares problem, checked against scipy's NNLS solver, against a brute-force
  scan of the objective, and on the closed cases (exact proportionality,
  anti-correlation, all-zero x, units outside every class).
- ebar (Eq. app-risk-score): the mean over calibration microbatches.
- psi (Eq. app-risk-score): equals kappa * ebar * sum |omega| alpha of Eq.
  token-weighted-risk, formed from the exposure oracle's own pieces.
- sparsity (App. D.3): brute-force counts and a numpy sort for the top-k share;
  closed forms for equal coefficients and constant-reward groups.
"""
import math

import numpy as np
import pytest
import scipy.optimize

from paper_2609_33570_amd import workloads as wl


# ------------------------------------------------------------------------ y --
def test_grad_rel_err_closed_forms(orc):
    rng = np.random.default_rng(5)
    g = rng.standard_normal(1000).astype(np.float32)
    assert orc.grad_rel_err(g, g) == 0.0
    assert orc.grad_rel_err(2 * g, g) == 1.0  # ||2g - g|| / ||g||, exact in binary
    z = np.zeros(1000, dtype=np.float32)
    want = math.sqrt(float(np.sum(g.astype(np.float64) ** 2)) / 1e-30)
    assert orc.grad_rel_err(g, z) == pytest.approx(want, rel=1e-15)
    assert orc.grad_rel_err(z, z) == 0.0


def test_grad_rel_err_against_numpy(orc):
    rng = np.random.default_rng(6)
    a = rng.standard_normal(4097).astype(np.float32)
    b = (a + 1e-3 * rng.standard_normal(4097)).astype(np.float32)
    want = np.linalg.norm(a.astype(np.float64) - b) / np.linalg.norm(b.astype(np.float64))
    got = orc.grad_rel_err(a, b)
    assert got == pytest.approx(want, rel=1e-12)
    # a common power-of-two scaling changes nothing
    assert orc.grad_rel_err(a * 64, b * 64) == got


# -------------------------------------------------------------------- kappa --
def calib_inputs(nb, nu, seed):
    rng = np.random.default_rng(seed)
    e = rng.uniform(0.1, 2.0, (nb, nu)).astype(np.float32)
    r = rng.uniform(1e-3, 5e-2, (nb, nu)).astype(np.float32)
    y = rng.uniform(0.0, 1e-2, (nb, nu)).astype(np.float32)
    return e, r, y


def test_kappa_is_the_nnls_solution(orc):
    nb, nu, nc = 6, 40, 4
    e, r, y = calib_inputs(nb, nu, 7)
    cls = np.arange(nu) % nc
    kappa, _ = orc.calibrate(cls, e, r, y, nc)
    for c in range(nc):
        sel = cls == c
        x = (e[:, sel].astype(np.float64) * r[:, sel]).ravel()
        t = y[:, sel].astype(np.float64).ravel()
        sol, _ = scipy.optimize.nnls(x[:, None], t)
        assert kappa[c] == pytest.approx(sol[0], rel=1e-10)
        # and it minimises the objective: no point of a fine scan does better
        obj = lambda k: np.sum((t - k * x) ** 2)  # noqa: E731
        scan = np.linspace(0, 3 * kappa[c] + 1e-9, 2001)
        assert obj(kappa[c]) <= min(obj(k) for k in scan) + 1e-18


def test_kappa_closed_cases(orc):
    nb, nu = 3, 8
    e, r, _ = calib_inputs(nb, nu, 8)
    x = e.astype(np.float64) * r
    cls = np.array([0, 0, 0, 1, 1, 2, -1, 7], dtype=np.int32)
    # class 0: y exactly proportional (kappa 2.5); class 1: anti-correlated -> 0;
    # class 2: x = 0 -> 0; units -1 and 7 belong to no class (n_classes = 3)
    y = np.zeros((nb, nu), dtype=np.float32)
    y[:, :3] = (2.5 * x[:, :3]).astype(np.float32)
    y[:, 3:5] = -x[:, 3:5].astype(np.float32)
    e2 = e.copy()
    e2[:, 5] = 0.0
    y[:, 6:] = 1e6  # would dominate any class they leaked into
    kappa, ebar = orc.calibrate(cls, e2, r, y, 3)
    assert kappa[0] == pytest.approx(2.5, rel=1e-7)  # y rounded to fp32
    assert kappa[1] == 0.0
    assert kappa[2] == 0.0
    np.testing.assert_allclose(ebar, r.astype(np.float64).mean(axis=0), rtol=1e-15)


def test_ebar_constant(orc):
    r = np.full((5, 3), 0.015625, dtype=np.float32)
    _, ebar = orc.calibrate(np.zeros(3, np.int32), np.ones((5, 3)), r, np.ones((5, 3)), 1)
    assert np.all(ebar == 0.015625)


# ---------------------------------------------------------------------- psi --
def test_psi_is_the_token_weighted_risk(orc):
    """Eq. app-risk-score (kappa E ebar) equals Eq. token-weighted-risk
    (kappa ebar sum_t |omega_t| alpha_t) with alpha from the row sums."""
    rows, cols = 64, 256
    x = wl.activation_host(rows, cols, seed=31, outliers=("channels", 0.02, 30.0))
    codes, scales = orc.quantize(x, orc.INT8, 64)
    ss_x, ss_e = orc.row_stats(x, orc.dequantize(codes, scales, orc.INT8, 64))
    rng = np.random.default_rng(9)
    w = rng.standard_normal(rows) * 1e-4
    mask = (rng.random(rows) > 0.25).astype(np.uint8)
    expo, _, _ = orc.unit_exposure_risk(w, mask, ss_x, ss_e, cols)
    kappa, ebar = np.array([0.75, 3.0]), np.array([0.02, 0.04])
    psi = orc.risk_score([1, 0], kappa, ebar, np.float32([expo, expo]))
    a = np.sqrt(ss_x / cols)
    valid = mask != 0
    alpha = (a + 1e-8) / (a[valid].mean() + 1e-8)
    direct = np.sum(np.abs(w[valid]) * alpha[valid])
    assert psi[0] == pytest.approx(3.0 * 0.02 * direct, rel=1e-6)  # exposure in fp32
    assert psi[1] == pytest.approx(0.75 * 0.04 * direct, rel=1e-6)


def test_psi_without_class_is_unavailable(orc):
    psi = orc.risk_score([0, -1, 2], [1.0, 2.0], [0.5, 0.5, 0.5], np.float32([1, 1, 1]))
    assert psi[0] == 0.5 and np.isinf(psi[1]) and np.isinf(psi[2])


# ----------------------------------------------------------------- sparsity --
def brute_sparsity(coeff, flags, adv, mask, R, T, frac):
    n = R * T
    valid = np.ones(n, bool) if mask is None else mask.astype(bool)
    advt = np.repeat(np.asarray(adv, np.float32), T)
    pad = int(np.sum(~valid))
    zero = int(np.sum(valid & (advt == 0)))
    clip = int(np.sum(valid & (advt != 0) & ((flags & 2) != 0)))
    mag = np.where(valid, np.abs(coeff), 0.0)
    k = max(1, math.ceil(frac * n))
    tot = mag.sum()
    share = np.sort(mag)[::-1][:k].sum() / tot if tot > 0 else 0.0
    return np.array([pad, zero, clip]), share


@pytest.mark.parametrize("pad_frac,beta,sigma", [(0.0, 0.0, 0.05), (0.3, 0.0, 0.25),
                                                 (0.3, 1e-3, 0.25)])
def test_sparsity_against_brute_force(orc, pad_frac, beta, sigma):
    P, G, T = 4, 8, 48
    b = wl.grpo_batch(P, G, T, seed=41, pad_frac=pad_frac, delta_sigma=sigma,
                      with_ref=beta > 0)
    adv, _, flags, coeff = orc.grpo_coeffs(b.rewards, b.logp_new, b.logp_old, b.logp_ref, b.mask,
                                           P, G, T, beta=beta)
    counts, share = orc.update_sparsity(coeff, flags, adv, b.mask, P * G, T, 0.1)
    want_c, want_s = brute_sparsity(coeff, flags, adv, b.mask, P * G, T, 0.1)
    np.testing.assert_array_equal(counts, want_c)
    assert share == pytest.approx(want_s, rel=1e-12)
    assert counts.sum() <= P * G * T


def test_sparsity_closed_forms(orc):
    R, T = 6, 10
    n = R * T
    # equal |omega| on the valid slots: the top-k share is min(k, n_valid) / n_valid
    mask = np.ones(n, np.uint8)
    mask[:15] = 0
    coeff = np.where(mask != 0, -0.125, 0.0)
    adv = np.ones(R, np.float32)
    counts, share = orc.update_sparsity(coeff, np.zeros(n, np.uint8), adv, mask, R, T, 0.1)
    assert list(counts) == [15, 0, 0]
    assert share == pytest.approx(6 / 45, rel=1e-15)
    # constant-reward groups: every valid slot has zero advantage; with beta = 0
    # every coefficient is 0 and the share is defined as 0
    P, G, T = 2, 4, 8
    rewards = np.ones(P * G, np.float32)
    lp = np.full(P * G * T, -2.0, np.float32)
    a, _, f, w = orc.grpo_coeffs(rewards, lp, lp, None, None, P, G, T)
    counts, share = orc.update_sparsity(w, f, a, None, P * G, T, 0.1)
    assert list(counts) == [0, P * G * T, 0] and share == 0.0
