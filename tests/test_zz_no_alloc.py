"""hilore_unit_exposure_risk_noalloc, the allocation-free variant of the
exposure/risk reduction (its partial sums in the library's fixed device
array), against the workspace entry point on the same inputs: both run the
same kernels in the same order, so every output must agree bit for bit.  Two
calls in a row, the second on a smaller input (fewer units, fewer rows), so
the second reuses the array the first left behind; a request beyond the
array's size is refused before anything is enqueued."""
import numpy as np
import pytest
import torch

from paper_2609_33570_amd import workloads as wl
from gpu_util import assert_bytes_equal, dev, filled, host

pytestmark = pytest.mark.gpu


def microbatch(hl, rows, n_units, seed):
    """GPU coefficients (30% padded) and GPU row sums of n_units compressed units."""
    b = wl.grpo_batch(1, 8, rows // 8, seed=seed, pad_frac=0.3, delta_sigma=0.1)
    adv = torch.empty(8, device="cuda")
    flags = torch.empty(rows, dtype=torch.uint8, device="cuda")
    coeff = torch.empty(rows, device="cuda")
    mask = dev(b.mask)
    hl.hilore_grpo_coeffs(dev(b.rewards), dev(b.logp_new), dev(b.logp_old), None, mask, 1, 8,
                          rows // 8, 0.2, 1e-6, 0.0, 0.0, adv, None, flags, coeff)
    keep, units = [], []
    for i in range(n_units):
        cols = 256 * (1 + i % 4)
        x = wl.activation_device(rows, cols, seed * 100 + i, outliers=("channels", 0.005, 30.0))
        codes = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
        scales = torch.empty((rows, cols // 128), device="cuda")
        ssx = torch.empty(rows, device="cuda")
        sse = torch.empty(rows, device="cuda")
        keep.append((x, codes, scales, ssx, sse))
        units.append(hl.unit_desc(x=x, codes=codes, scales=scales, row_ss_x=ssx, row_ss_err=sse))
    hl.hilore_compress(units, 1, 128)
    return coeff, mask, units, keep


def both(hl, coeff, mask, rows, units):
    n = len(units)
    ref = [filled(n, torch.float32, float("nan")) for _ in range(3)]
    got = [filled(n, torch.float32, float("nan")) for _ in range(3)]
    ws = torch.empty(hl.hilore_unit_exposure_risk_workspace_bytes(rows, n), dtype=torch.uint8,
                     device="cuda")
    hl.hilore_unit_exposure_risk(coeff, mask, rows, units, 1e-8, 1e-8, *ref, workspace=ws)
    hl.hilore_unit_exposure_risk_noalloc(coeff, mask, rows, units, 1e-8, 1e-8, *got)
    torch.cuda.synchronize()
    return [host(t) for t in ref], [host(t) for t in got]


def test_noalloc_matches_workspace_entry_point(hl):
    # first call: 40 units x 10240 rows (200 partial slots); second: 6 units x
    # 3000 rows (ragged, 12 slots), over what the first left in the array
    for rows, n_units, seed in ((10240, 40, 61), (3000, 6, 62)):
        coeff, mask, units, keep = microbatch(hl, rows, n_units, seed)
        ref, got = both(hl, coeff, mask, rows, units)
        for name, r, g in zip(("exposure", "risk", "rel_err"), ref, got):
            assert np.isfinite(r).all(), name
            assert_bytes_equal(g, r, f"{name} ({n_units} units x {rows} rows)")
        assert (ref[0] > 0).all() and (ref[1] > 0).all()


def test_noalloc_refuses_more_than_its_array(hl):
    """5 units of 2^24 - 1 rows need 5 x 8192 x 32 B = 1.25 MiB of partials, more
    than the 1 MiB array: refused with HILORE_ERR_WORKSPACE before anything is
    launched (which is why the buffers may be tiny here)."""
    rows = (1 << 24) - 1
    small = torch.empty(16, device="cuda")
    units = [hl.unit_desc(row_ss_x=small, row_ss_err=small, rows=rows, cols=128)
             for _ in range(5)]
    outs = [torch.empty(5, device="cuda") for _ in range(3)]
    with pytest.raises(hl.HiloreError) as e:
        hl.hilore_unit_exposure_risk_noalloc(small, None, rows, units, 1e-8, 1e-8, *outs)
    assert e.value.status == hl.HILORE_ERR_WORKSPACE
    # at the limit: 4 units x 8192 chunks fit exactly (not launched here)
    assert hl.hilore_unit_exposure_risk_workspace_bytes(rows, 4) == 1 << 20
