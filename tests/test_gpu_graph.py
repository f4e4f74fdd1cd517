"""The hot path captured in a HIP graph (through torch.cuda.graph): the calls
allocate nothing (the exposure/risk workspace is the caller's), record no
memset and never synchronise the host, so one step (coefficients, compress
with row sums, exposure and risk, decompress, the fused wgrad) captures as is.  The graph is replayed three times with new
inputs written eagerly in between, and every replay must equal the same step
run eagerly on the same inputs, bit for bit."""
import numpy as np
import pytest
import torch

from paper_2609_33570_amd import workloads as wl
from gpu_util import assert_bytes_equal, dev, host

pytestmark = pytest.mark.gpu

P, G, T = 1, 8, 256
ROWS = P * G * T
COLS, BLOCK, CODE = 1536, 128, 1
K, M, N = 2048, 512, 256


def buffers(hl):
    b = {"rewards": torch.empty(P * G, device="cuda"), "lp_new": torch.empty(ROWS, device="cuda"),
         "lp_old": torch.empty(ROWS, device="cuda"), "adv": torch.empty(P * G, device="cuda"),
         "ratio": torch.empty(ROWS, device="cuda"),
         "flags": torch.empty(ROWS, dtype=torch.uint8, device="cuda"),
         "coeff": torch.empty(ROWS, device="cuda"),
         "x": torch.empty((ROWS, COLS), dtype=torch.bfloat16, device="cuda"),
         "codes": torch.empty((ROWS, COLS), dtype=torch.uint8, device="cuda"),
         "scales": torch.empty((ROWS, COLS // BLOCK), device="cuda"),
         "xhat": torch.empty((ROWS, COLS), dtype=torch.bfloat16, device="cuda"),
         "ssx": torch.empty(ROWS, device="cuda"), "sse": torch.empty(ROWS, device="cuda"),
         "expo": torch.empty(1, device="cuda"), "risk": torch.empty(1, device="cuda"),
         "rel": torch.empty(1, device="cuda"),
         "wc": torch.empty((K, M), dtype=torch.uint8, device="cuda"),
         "ws": torch.empty((K, M // BLOCK), device="cuda"),
         "dy": torch.empty((K, N), dtype=torch.bfloat16, device="cuda"),
         "dw": torch.empty((M, N), device="cuda"),
         "risk_ws": torch.empty(hl.hilore_unit_exposure_risk_workspace_bytes(ROWS, 1),
                                dtype=torch.uint8, device="cuda")}
    b["unit"] = hl.unit_desc(x=b["x"], codes=b["codes"], scales=b["scales"], xhat=b["xhat"],
                             row_ss_x=b["ssx"], row_ss_err=b["sse"])
    return b


def load_inputs(hl, b, seed):
    """New inputs written eagerly into the captured buffers."""
    g = wl.grpo_batch(P, G, T, seed=seed)
    b["rewards"].copy_(dev(g.rewards))
    b["lp_new"].copy_(dev(g.logp_new))
    b["lp_old"].copy_(dev(g.logp_old))
    b["x"].copy_(wl.activation_device(ROWS, COLS, seed + 1, outliers=("channels", 0.005, 30.0)))
    xw = wl.activation_device(K, M, seed + 2)
    hl.hilore_compress([hl.unit_desc(x=xw, codes=b["wc"], scales=b["ws"])], CODE, BLOCK)
    b["dy"].copy_(wl.normal_bf16_device(K, N, seed + 3, 0.02))
    torch.cuda.synchronize()


def step(hl, b):
    hl.hilore_grpo_coeffs(b["rewards"], b["lp_new"], b["lp_old"], None, None, P, G, T, 0.2, 1e-6,
                          0.0, 0.0, b["adv"], b["ratio"], b["flags"], b["coeff"])
    hl.hilore_compress([b["unit"]], CODE, BLOCK)
    hl.hilore_unit_exposure_risk(b["coeff"], None, ROWS, [b["unit"]], 1e-8, 1e-8, b["expo"],
                                 b["risk"], b["rel"], workspace=b["risk_ws"])
    hl.hilore_decompress([b["unit"]], CODE, BLOCK)
    hl.hilore_dequant_wgrad(b["wc"], b["ws"], CODE, BLOCK, b["dy"], b["dw"], K, M, N)


OUT = ("adv", "ratio", "flags", "coeff", "codes", "scales", "xhat", "ssx", "sse", "expo", "risk",
       "rel", "dw")


def snapshot(b):
    return {k: host(b[k]) for k in OUT}


def test_graph_replays_match_eager(hl):
    b = buffers(hl)
    load_inputs(hl, b, 3000)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(hl, b)  # warm-up off the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(hl, b)
    for r, seed in enumerate((3100, 3200, 3300)):
        load_inputs(hl, b, seed)
        graph.replay()
        torch.cuda.synchronize()
        got = snapshot(b)
        for k in OUT:  # scribble over the outputs, then the eager step rewrites them
            b[k].view(torch.uint8).fill_(0xA5)
        step(hl, b)
        torch.cuda.synchronize()
        want = snapshot(b)
        for k in OUT:
            assert_bytes_equal(got[k], want[k], f"replay {r}: {k}")
        assert np.isfinite(want["dw"]).all() and want["expo"][0] > 0
