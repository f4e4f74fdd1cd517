"""GPU parity of hilore_unit_exposure_risk, run on the GPU's own coefficients
and row sums, against the oracle's fp64 truth built from the same inputs."""
import numpy as np
import pytest
import torch

from paper_2609_33570_amd import workloads as wl
from gpu_util import assert_close, dev, filled, host

pytestmark = pytest.mark.gpu


def gpu_pipeline(hl, b, xs, code, block, beta=0.0):
    """GRPO coefficients, batched compress with row sums, then the per-unit
    reduction, all on one stream, like one microbatch of the hot path."""
    R, n = b.P * b.G, b.P * b.G * b.T
    adv = filled(R, torch.float32, 0)
    flags = filled(n, torch.uint8, 0)
    coeff = filled(n, torch.float32, float("nan"))
    m = dev(b.mask) if b.mask is not None else None
    hl.hilore_grpo_coeffs(dev(b.rewards), dev(b.logp_new), dev(b.logp_old),
                          dev(b.logp_ref) if b.logp_ref is not None else None, m, b.P, b.G, b.T,
                          0.2, 1e-6, beta, 0.0, adv, None, flags, coeff)
    units, keep = [], []
    for x in xs:
        rows, cols = x.shape
        xd = dev(x)
        codes = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
        scales = torch.empty((rows, cols // block), dtype=torch.float32, device="cuda")
        ssx = filled(rows, torch.float32, float("nan"))
        sse = filled(rows, torch.float32, float("nan"))
        keep.append((xd, codes, scales, ssx, sse))
        units.append(hl.unit_desc(x=xd, codes=codes, scales=scales, row_ss_x=ssx, row_ss_err=sse))
    hl.hilore_compress(units, code, block)
    k = len(xs)
    expo = filled(k, torch.float32, float("nan"))
    risk = filled(k, torch.float32, float("nan"))
    rel = filled(k, torch.float32, float("nan"))
    hl.hilore_unit_exposure_risk(coeff, m, n, units, 1e-8, 1e-8, expo, risk, rel)
    torch.cuda.synchronize()
    return host(expo), host(risk), host(rel)


def oracle_pipeline(orc, b, xs, code, block, beta=0.0):
    _, _, _, coeff = orc.grpo_coeffs(b.rewards, b.logp_new, b.logp_old, b.logp_ref, b.mask,
                                     b.P, b.G, b.T, beta=beta)
    out = []
    for x in xs:
        codes, scales = orc.quantize(x, code, block)
        xh = orc.dequantize(codes, scales, code, block)
        ss_x, ss_e = orc.row_stats(x, xh)
        out.append(orc.unit_exposure_risk(coeff, b.mask, ss_x, ss_e, x.shape[1]))
    return [np.array(v) for v in zip(*out)]


@pytest.mark.parametrize("code,block", [(0, 64), (1, 128)], ids=["int8-64", "e4m3fn-128"])
@pytest.mark.parametrize("pad", [None, 0.3])
@pytest.mark.parametrize("beta", [0.0, 1e-3])
def test_units_of_a_microbatch(hl, orc, code, block, pad, beta):
    b = wl.grpo_batch(2, 8, 256, seed=41, with_ref=beta > 0, pad_frac=pad, delta_sigma=0.1)
    rows = b.P * b.G * b.T
    xs = [wl.activation_host(rows, c, seed=300 + i, outliers=("channels", 0.005, 30.0))
          for i, c in enumerate([256, 512, 1024, 768, 1536])]
    g = gpu_pipeline(hl, b, xs, code, block, beta)
    o = oracle_pipeline(orc, b, xs, code, block, beta)
    for name, gv, ov in zip(["exposure", "risk", "rel_err"], g, o):
        assert_close(gv, ov, name)


def test_many_units_and_empty_token_set(hl, orc):
    b = wl.grpo_batch(1, 8, 128, seed=42, pad_frac=0.4)
    rows = 1024
    xs = [wl.activation_host(rows, 128, seed=400 + i) for i in range(40)]
    g = gpu_pipeline(hl, b, xs, 0, 64)
    o = oracle_pipeline(orc, b, xs, 0, 64)
    for name, gv, ov in zip(["exposure", "risk", "rel_err"], g, o):
        assert_close(gv, ov, name)
    b.mask[:] = 0
    g = gpu_pipeline(hl, b, xs[:3], 0, 64)
    assert (g[0] == 0).all() and (g[1] == 0).all() and (g[2] > 0).all()


def test_deterministic(hl, orc):
    """Fixed-order sums: the whole chain (coefficients, compress with row sums,
    exposure and risk) run twice on the same inputs agrees bit for bit."""
    b = wl.grpo_batch(2, 8, 512, seed=43, pad_frac=0.2, delta_sigma=0.1)
    rows = b.P * b.G * b.T
    xs = [wl.activation_host(rows, c, seed=500 + i) for i, c in enumerate([1024, 2048, 3584])]
    first = gpu_pipeline(hl, b, xs, 1, 128)
    second = gpu_pipeline(hl, b, xs, 1, 128)
    for name, a1, a2 in zip(["exposure", "risk", "rel_err"], first, second):
        assert np.array_equal(a1.view(np.uint32), a2.view(np.uint32)), name


def risk_on(hl, orc, coeff, mask, xs, code, block, workspace=None):
    """GPU: compress with row sums, then the reduction on the given coefficients;
    oracle: the same from its own codec, in fp64."""
    rows = coeff.size
    units, keep = [], []
    for x in xs:
        xd = dev(x)
        codes = torch.empty(x.shape, dtype=torch.uint8, device="cuda")
        scales = torch.empty((x.shape[0], x.shape[1] // block), dtype=torch.float32, device="cuda")
        ssx = filled(rows, torch.float32, float("nan"))
        sse = filled(rows, torch.float32, float("nan"))
        keep.append((xd, codes, scales, ssx, sse))
        units.append(hl.unit_desc(x=xd, codes=codes, scales=scales, row_ss_x=ssx, row_ss_err=sse))
    hl.hilore_compress(units, code, block)
    k = len(xs)
    outs = [filled(k, torch.float32, float("nan")) for _ in range(3)]
    m = dev(mask) if mask is not None else None
    hl.hilore_unit_exposure_risk(dev(coeff), m, rows, units, 1e-8, 1e-8, *outs,
                                 workspace=workspace)
    torch.cuda.synchronize()
    want = []
    for x in xs:
        c, s = orc.quantize(x, code, block)
        ss_x, ss_e = orc.row_stats(x, orc.dequantize(c, s, code, block))
        want.append(orc.unit_exposure_risk(coeff.astype(np.float64), mask, ss_x, ss_e, x.shape[1]))
    return [host(o) for o in outs], [np.array(v) for v in zip(*want)]


def random_coeff(rows, seed, pad=0.3):
    g = np.random.default_rng(seed)
    mask = (g.random(rows) >= pad).astype(np.uint8)
    coeff = (g.normal(0.0, 1e-4, rows) * mask).astype(np.float32)
    return coeff, mask


@pytest.mark.parametrize("rows", [1, 3, 2048, 2049, 7171], ids=lambda r: f"rows{r}")
def test_ragged_row_counts(hl, orc, rows):
    """Chunks of 2048 rows read as runs of 4: one and three rows (tail only), a
    whole chunk, one past it, and 3 chunks plus a tail of 1027 rows."""
    coeff, mask = random_coeff(rows, 700 + rows)
    xs = [wl.activation_host(rows, c, seed=710 + i, outliers=("channels", 0.005, 30.0))
          for i, c in enumerate([128, 384])]
    got, want = risk_on(hl, orc, coeff, mask, xs, 1, 128)
    for name, gv, ov in zip(["exposure", "risk", "rel_err"], got, want):
        assert_close(gv, ov, f"{name} rows={rows}")


def test_more_units_than_one_launch(hl, orc):
    """100 units: two partial launches (96 units travel in one launch's
    arguments) and one fold; an explicit workspace of exactly the queried size."""
    rows = 2100
    coeff, mask = random_coeff(rows, 720)
    xs = [wl.activation_host(rows, 64 * (1 + i % 3), seed=730 + i) for i in range(100)]
    nbytes = hl.hilore_unit_exposure_risk_workspace_bytes(rows, len(xs))
    assert nbytes == 100 * 2 * 32
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    got, want = risk_on(hl, orc, coeff, mask, xs, 0, 64, workspace=ws)
    for name, gv, ov in zip(["exposure", "risk", "rel_err"], got, want):
        assert_close(gv, ov, name)


def test_no_rows(hl):
    """rows = 0: nothing to read and no workspace; exposure and risk 0, rel_err
    0 / (0 + eps) = 0."""
    outs = [filled(2, torch.float32, float("nan")) for _ in range(3)]
    d = [hl.unit_desc(rows=0, cols=128), hl.unit_desc(rows=0, cols=64)]
    hl.hilore_unit_exposure_risk(None, None, 0, d, 1e-8, 1e-8, *outs)
    torch.cuda.synchronize()
    for o in outs:
        assert (host(o) == 0).all()
