"""Pins of the oracle's H/L/R allocation (Sec. 3.4 Eq. joint-allocation,
solved by the dynamic programme of App. B.2 on the conservative grid of Eqs.
allocation-grid / allocation-integer-costs).

  - against exhaustive enumeration of all 3^U assignments of the same
    discretised problem (U <= 9): optimum, terminal costs and a valid optimal
    assignment; with integer utilities (exact sums, many ties) the whole
    assignment, tie rules included;
  - against an independent integer-programming solver (scipy's HiGHS MILP) on
    larger instances (U up to 60);
  - the grid's feasibility guarantee (Eq. allocation-grid-feasibility), the
    available-action rule (Eq. available-recovery-actions), the exclusion of
    non-positive utilities, and the zero-budget boundary cases.
"""
import numpy as np
import pytest
import scipy.optimize as so

from paper_2609_33570_amd import workloads as wl


def costs(inst, n_b, n_d):
    """Integer costs and availability, recomputed here from the definitions."""
    U = inst.U
    ok = np.zeros((U, 3), bool)
    b = np.zeros((U, 3), np.int64)
    r = np.zeros((U, 3), np.int64)
    tau = np.zeros((U, 3))
    ok[:, 0] = True
    for u in range(U):
        for a, t, dm, rk in ((1, inst.tau_h[u], inst.dm_h[u], 0.0),
                             (2, inst.tau_l[u], inst.dm_l[u], inst.psi[u])):
            allowed = {1: (1, 2), 2: (2,)}.get(int(inst.q[u]), ())
            if a not in allowed or not (inst.verified[u] >> a) & 1 or not t > 0:
                continue
            if a == 2 and inst.delta_b == 0:
                continue
            bb = np.ceil(dm / (inst.m_res / n_b)) if inst.m_res > 0 else (0 if dm == 0 else n_b + 1)
            rr = (np.ceil(rk / (inst.delta_b / n_d)) if inst.delta_b > 0 else 0) if a == 2 else 0
            if bb <= n_b and rr <= n_d:
                ok[u, a], b[u, a], r[u, a], tau[u, a] = True, bb, rr, t
    return ok, b, r, tau


def check_assignment(inst, act, totals, jk, n_b, n_d):
    ok, b, r, tau = costs(inst, n_b, n_d)
    u = np.arange(inst.U)
    assert ok[u, act].all(), "chosen action not available"
    assert b[u, act].sum() == jk[0] <= n_b and r[u, act].sum() == jk[1] <= n_d
    v = 0.0
    for i in range(inst.U):
        if act[i]:
            v += tau[i, act[i]]
    assert v == totals[0]
    # Eq. allocation-grid-feasibility: the real costs fit the real budgets
    mem = np.where(act == 1, inst.dm_h, np.where(act == 2, inst.dm_l, 0.0)).sum()
    risk = np.where(act == 2, inst.psi, 0.0).sum()
    assert mem <= inst.m_res * (1 + 1e-12) + 1e-300
    assert risk <= inst.delta_b * (1 + 1e-12) + 1e-300
    np.testing.assert_allclose(totals[1:], [mem, risk], rtol=1e-12)


@pytest.mark.parametrize("seed", range(40))
def test_dp_equals_enumeration(orc, seed):
    g = np.random.default_rng(seed)
    U = int(g.integers(1, 10))
    n_b, n_d = [(8, 8), (16, 32), (1024, 1024), (5, 200)][seed % 4]
    inst = wl.alloc_small(U, seed)
    a1, t1, jk1 = orc.allocate(*inst.arrays(), inst.m_res, inst.delta_b, n_b, n_d)
    a2, t2, jk2 = orc.allocate(*inst.arrays(), inst.m_res, inst.delta_b, n_b, n_d, brute=True)
    assert t1[0] == t2[0] and np.array_equal(jk1, jk2)
    check_assignment(inst, a1, t1, jk1, n_b, n_d)


@pytest.mark.parametrize("seed", range(40))
def test_dp_equals_enumeration_with_ties(orc, seed):
    """Integer utilities: every partial sum is exact, so the DP's tie rules
    (terminal: lower risk, then memory; within a state R, H, L) must select
    exactly the enumeration's assignment."""
    g = np.random.default_rng(100 + seed)
    U = int(g.integers(1, 10))
    inst = wl.alloc_small(U, 100 + seed, integer=True, scale=4.0)
    a1, t1, jk1 = orc.allocate(*inst.arrays(), inst.m_res, inst.delta_b, 8, 8)
    a2, t2, jk2 = orc.allocate(*inst.arrays(), inst.m_res, inst.delta_b, 8, 8, brute=True)
    assert np.array_equal(a1, a2) and np.array_equal(t1, t2) and np.array_equal(jk1, jk2)


@pytest.mark.parametrize("U,n,seed", [(30, 64, 1), (45, 128, 2), (60, 1024, 3), (60, 256, 4)])
def test_dp_equals_milp(orc, U, n, seed):
    inst = wl.alloc_small(U, 200 + seed)
    act, tot, jk = orc.allocate(*inst.arrays(), inst.m_res, inst.delta_b, n, n)
    check_assignment(inst, act, tot, jk, n, n)
    ok, b, r, tau = costs(inst, n, n)
    idx = [(u, a) for u in range(U) for a in range(3) if ok[u, a]]
    c = -np.array([tau[u, a] for u, a in idx])
    A_one = np.zeros((U, len(idx)))
    for k, (u, a) in enumerate(idx):
        A_one[u, k] = 1
    A_b = np.array([[b[u, a] for u, a in idx]], float)
    A_r = np.array([[r[u, a] for u, a in idx]], float)
    res = so.milp(c, integrality=np.ones(len(idx)), bounds=so.Bounds(0, 1),
                  constraints=[so.LinearConstraint(A_one, 1, 1), so.LinearConstraint(A_b, -np.inf, n),
                               so.LinearConstraint(A_r, -np.inf, n)],
                  options={"mip_rel_gap": 0.0})
    assert res.status == 0
    np.testing.assert_allclose(tot[0], -res.fun, rtol=1e-9)


def test_boundary_cases(orc):
    inst = wl.alloc_small(8, 7)
    arrs = list(inst.arrays())
    # only R retained -> nothing but R, zero utility
    q_r = np.zeros(8, np.uint8)
    a, t, jk = orc.allocate(q_r, *arrs[1:], inst.m_res, inst.delta_b)
    assert (a == 0).all() and t[0] == 0 and (jk == 0).all()
    # zero risk budget disables L; zero memory budget admits only zero-memory actions
    a, t, jk = orc.allocate(*arrs, inst.m_res, 0.0)
    assert (a != 2).all() and jk[1] == 0
    a, t, jk = orc.allocate(*arrs, 0.0, inst.delta_b)
    dm = np.where(a == 1, inst.dm_h, np.where(a == 2, inst.dm_l, 0.0))
    assert (dm == 0).all() and jk[0] == 0
    # budgets that never bind: every unit independently takes its best action
    # (R < H < L on equal utility), utilities > 0 only
    a, t, jk = orc.allocate(*arrs, 1e30, 1e30)
    for u in range(8):
        allowed = {1: (1, 2), 2: (2,)}.get(int(inst.q[u]), ())
        cand = [(0.0, 0)] + [(tt, k) for k, tt in ((1, inst.tau_h[u]), (2, inst.tau_l[u]))
                             if k in allowed and (inst.verified[u] >> k) & 1 and tt > 0]
        best = max(cand, key=lambda x: (x[0], -x[1]))
        assert a[u] == best[1]
    # an L copy cannot give H; an unverified action is never taken
    q_l = np.full(8, 2, np.uint8)
    a, _, _ = orc.allocate(q_l, *arrs[1:], 1e30, 1e30)
    assert (a != 1).all()
    ver = np.full(8, 0b011, np.uint8)
    a, _, _ = orc.allocate(arrs[0], ver, *arrs[2:], 1e30, 1e30)
    assert (a != 2).all()
    with pytest.raises(ValueError):
        orc.allocate(*arrs, -1.0, 1.0)
