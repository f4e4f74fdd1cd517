"""Benchmark of the HiLoRe hot path on one MI355X.

One step = one pass of the whole hot path over one microbatch of the
Qwen2-7B-width layer workload (8 responses x 2048 tokens = 16384 rows), in the
order of Algorithm 1:
  1. hilore_grpo_coeffs        GRPO coefficients for the 16384 token slots
  2. hilore_compress           hidden 16384x3584 + MLP 16384x18944 -> fp8-e4m3 1x128,
                               with per-row sums (one batched call)
  3. hilore_unit_exposure_risk exposure / risk / relative error of both units
  4. hilore_decompress         both units back to bf16 (one batched call)
  5. hilore_dequant_wgrad      dW 4096x4096 = deq(X)^T dY, X fp8-e4m3 1x128
                               16384x4096, dY bf16 16384x4096 (fp32 accumulate)
Inputs are synthetic (seeded, drawn on the device) and resident in HBM before
the timed region; four buffer sets are rotated so that consecutive steps do
not hit the 256 MB infinity cache with the previous step's data.

Prints ONE JSON line.  `value` is compress+decompress throughput in GB/s of
algorithmic bytes (the first figure of the metric); the wgrad TFLOP/s and the
coefficient tokens/s ride along, each with its own roofline.  Every duration
is the median over the timed steps of HIP events recorded around the call on
the stream it runs on (the mean rides along).

`configs` holds the other workloads, each timed the same way after the step:
  tiny               coefficient and codec latency (1024 slots; 1024x896 int8 1x128)
  qwen2_7b_plan      78 L units of 16384x3584, int8 1x64: batched compress with row
                     sums, exposure/risk, batched decompress
  llama3_8b_stress   32 units of 32768x14336 Student-t, int8 1x128, 30% padded GRPO
                     batch; coefficients also at the literal 65536 slots
and `coeff_sweep` the coefficients on 2^20 .. 2^26 masked slots with N counted.
For context the line also times hilore_allocate (the H/L/R dynamic programme
that follows the exposure step) on a 196-unit plan and, under "next", the
calls that follow the five rows (the LoRA adapter gradient and the gated-MLP
activation backward on the MLP unit, the calibration scalars, the
update-sparsity diagnostics), all outside the step; `cpu_baseline` times the
CPU oracle on the host on bounded samples of the same workloads.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

from paper_2609_33570_amd import defaults as D

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "compress+decompress GB/s (% HBM peak); fused dequant-wgrad TFLOP/s; coeff tok/s"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
N_SETS = 4
SWEEP_G, SWEEP_T, SWEEP_PAD = 16, 1024, 0.3


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--step-only", action="store_true",
                   help="time only the layer step (no other configs, sweep or context calls)")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a plain 1 GiB device copy (for scaling HBM byte counters)")
    p.add_argument("--blas-ref", action="store_true",
                   help="also time hipBLASLt's bf16 GEMM (torch.mm) on the reconstructed X, for context")
    p.add_argument("--sweep-max-log2", type=int, default=26,
                   help="largest coefficient-sweep size, as log2 of the slot count")
    return p.parse_args()


def progress(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def codec_bytes(rows, cols, block, stats):
    """Algorithmic HBM bytes of one compress and one decompress of a unit:
    read bf16 x, write codes + scales (+ two fp32 row sums); read codes +
    scales, write bf16 xhat."""
    n = rows * cols
    scales = 4 * n // block
    comp = 2 * n + n + scales + (8 * rows if stats else 0)
    decomp = n + scales + 2 * n
    return comp, decomp


def grpo_bytes(slots, responses, masked):
    """Algorithmic bytes of one coefficient call (beta = 0, ratio written):
    logp_new and logp_old read, coeff and ratio written (4 B each), flags
    written and the mask read (1 B each), reward read and advantage written per
    response."""
    return slots * (16 + 1 + (1 if masked else 0)) + responses * 8


def risk_bytes(rows, units, masked):
    """Both fp32 row sums of every unit, the coefficients and the mask once."""
    return rows * 8 * units + rows * (4 + (1 if masked else 0))


KERNEL_SOURCES = {"compress": ["codec.hip"], "decompress": ["codec.hip"],
                  "dequant_wgrad": ["wgrad.hip"], "grpo_coeffs": ["grpo.hip"],
                  "exposure_risk": ["risk.hip"], "dequant_lora_grad": ["lora.hip"],
                  "dequant_lora_grad_5": ["lora.hip"],
                  "grad_rel_err": ["calib.hip"], "dequant_swiglu_bwd": ["swiglu.hip"],
                  "allocate_dp": ["alloc.hip"]}


def measured_traffic():
    """HBM bytes per call ("<workload>/<kernel>") from the committed rocprofv3
    counter summary, for the kernels whose sources are unchanged since the
    counters were taken (else None)."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(path):
        return {}
    table = json.load(open(path))
    csrc = os.path.join(ROOT, "paper_2609_33570_amd", "csrc")
    common = ["device_common.hpp", "hilore_internal.hpp"]
    out = {}
    for key, ent in table.get("kernels", {}).items():
        h = hashlib.sha256()
        for f in KERNEL_SOURCES.get(key.split("/")[-1], []) + common:
            with open(os.path.join(csrc, f), "rb") as fh:
                h.update(fh.read())
        out[key] = ent["traffic_bytes"] if h.hexdigest() == ent["source_sha256"] else None
    return out


TRAFFIC = {}


def roof(workload, name, per_call, ms, peak=HBM_PEAK_GBS, unit="GB/s", bound="hbm",
         what=None):
    """Roofline entry of one kernel call: `per_call` algorithmic bytes (or
    FLOP) over the call's median duration `ms`."""
    scale = 1e9 if unit == "GB/s" else 1e12
    a = per_call / (ms * 1e-3) / scale
    return {"kernel": name, "bound": bound, "achieved": round(a, 2), "peak": peak, "unit": unit,
            "frac": round(a / peak, 4), "us": round(ms * 1e3, 2),
            "traffic": TRAFFIC.get(f"{workload}/{name}"),
            "algorithmic": what or f"{per_call} {'B' if unit == 'GB/s' else 'FLOP'} per call"}


def timed_steps(step, n_calls, steps, warmup, n_sets=1):
    """Run `warmup` untimed and `steps` timed steps; step(i, mark) records
    mark(k) before call k and mark(n_calls) after the last.  Returns the
    per-call durations (ms, one list per call) and the wall time per step."""
    import torch

    for i in range(warmup):
        step(i % n_sets, None)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n_calls + 1)]
           for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        ev = evs[i]
        step(i % n_sets, lambda k, ev=ev: ev[k].record())
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / max(steps, 1)
    per = [[ev[k].elapsed_time(ev[k + 1]) for ev in evs] for k in range(n_calls)]
    return per, wall


def graph_us(call, n_sets=1, n_calls=20, replays=5):
    """Per-call GPU time (us) of call(i) with n_calls calls captured in one HIP
    graph (through torch.cuda.graph) and the graph replayed: the kernels run
    back to back with no host work between them, which is how a latency-bound
    call runs inside a captured training step.  Eager per-call events of such
    calls measure the host's submission instead."""
    import torch

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for i in range(2):
            call(i % n_sets)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(n_calls):
            call(i % n_sets)
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(replays):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (replays * n_calls)
    del g
    return round(us, 2)


def med(v):
    return statistics.median(v)


def us_stats(v):
    return {"median": round(med(v) * 1e3, 2), "mean": round(statistics.fmean(v) * 1e3, 2)}


def host_bf16(t):
    import numpy as np
    import torch

    return t.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


# ----------------------------------------------------------------- layer step --
def layer_step(args, hl, wl):
    """The headline step: Qwen2-7B-width layer codec path + the 4096^3 wgrad."""
    import torch

    w = wl.QWEN2_7B_LAYER
    ww = wl.WGRAD_4096
    code, block = hl.HILORE_CODE_FP8_E4M3FN, 128
    K, M, N = ww.wgrad
    R = w.P * w.G
    rows = R * w.T
    b = wl.grpo_batch(w.P, w.G, w.T, seed=w.seed)

    progress("drawing the layer step's inputs on the device")
    sets = []
    for s in range(N_SETS):
        st = {"grpo_host": b}
        st["rewards"], st["lp_new"], st["lp_old"] = (torch.from_numpy(a).cuda() for a in
                                                     (b.rewards, b.logp_new, b.logp_old))
        st["adv"] = torch.empty(R, dtype=torch.float32, device="cuda")
        st["flags"] = torch.empty(rows, dtype=torch.uint8, device="cuda")
        st["coeff"] = torch.empty(rows, dtype=torch.float32, device="cuda")
        st["ratio"] = torch.empty(rows, dtype=torch.float32, device="cuda")
        units_c, units_d, keep = [], [], []
        for i, u in enumerate(w.units):
            x = wl.activation_device(u.rows, u.cols, w.seed * 10 + i + 1000 * s,
                                     outliers=w.outliers)
            codes = torch.empty((u.rows, u.cols), dtype=torch.uint8, device="cuda")
            scales = torch.empty((u.rows, u.cols // block), dtype=torch.float32, device="cuda")
            xhat = torch.empty((u.rows, u.cols), dtype=torch.bfloat16, device="cuda")
            ssx = torch.empty(u.rows, dtype=torch.float32, device="cuda")
            sse = torch.empty(u.rows, dtype=torch.float32, device="cuda")
            keep.append((x, codes, scales, xhat, ssx, sse))
            units_c.append(hl.unit_desc(x=x, codes=codes, scales=scales, row_ss_x=ssx,
                                        row_ss_err=sse))
            units_d.append(hl.unit_desc(codes=codes, scales=scales, xhat=xhat))
        st["keep"], st["uc"], st["ud"] = keep, units_c, units_d
        st["expo"] = torch.empty(len(w.units), dtype=torch.float32, device="cuda")
        st["risk"] = torch.empty_like(st["expo"])
        st["rel"] = torch.empty_like(st["expo"])
        st["risk_ws"] = torch.zeros(hl.hilore_unit_exposure_risk_workspace_bytes(rows, len(w.units)),
                                    dtype=torch.uint8, device="cuda")
        # wgrad operands: X stored as fp8-e4m3 1x128 (encoded here, outside the timed region)
        xw = wl.activation_device(K, M, ww.seed + 1000 * s)
        wc = torch.empty((K, M), dtype=torch.uint8, device="cuda")
        ws = torch.empty((K, M // block), dtype=torch.float32, device="cuda")
        hl.hilore_compress([hl.unit_desc(x=xw, codes=wc, scales=ws)], code, block)
        del xw
        st["wc"], st["ws"] = wc, ws
        st["dy"] = wl.normal_bf16_device(K, N, ww.seed + 100 + 1000 * s, 0.02)
        st["dw"] = torch.empty((M, N), dtype=torch.float32, device="cuda")
        sets.append(st)
    torch.cuda.synchronize()

    names = ["grpo_coeffs", "compress", "exposure_risk", "decompress", "dequant_wgrad"]

    def step(i, mark):
        st = sets[i]
        mark = mark or (lambda k: None)
        mark(0)
        hl.hilore_grpo_coeffs(st["rewards"], st["lp_new"], st["lp_old"], None, None, w.P, w.G,
                              w.T, D.CLIP_EPS, D.ADV_EPS, 0.0, 0.0, st["adv"], st["ratio"],
                              st["flags"], st["coeff"])
        mark(1)
        hl.hilore_compress(st["uc"], code, block)
        mark(2)
        hl.hilore_unit_exposure_risk(st["coeff"], None, rows, st["uc"], D.EPS_ALPHA, D.EPS_REL,
                                     st["expo"], st["risk"], st["rel"], workspace=st["risk_ws"])
        mark(3)
        hl.hilore_decompress(st["ud"], code, block)
        mark(4)
        hl.hilore_dequant_wgrad(st["wc"], st["ws"], code, block, st["dy"], st["dw"], K, M, N,
                                False)
        mark(5)

    if args.copy_calibration:
        # a plain copy of known size: 2^29 bf16 = 1 GiB read + 1 GiB written
        src = torch.ones(1 << 29, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    progress(f"layer step: {args.warmup} warm-up and {args.steps} timed steps")
    per, wall = timed_steps(step, len(names), args.steps, args.warmup, N_SETS)
    ms = {n: med(per[k]) for k, n in enumerate(names)}

    comp_b = decomp_b = 0
    for u in w.units:
        c, d = codec_bytes(u.rows, u.cols, block, stats=True)
        comp_b += c
        decomp_b += d
    codec_gbs = (comp_b + decomp_b) / ((ms["compress"] + ms["decompress"]) * 1e-3) / 1e9
    wflops = 2.0 * K * M * N
    wgrad_tflops = wflops / (ms["dequant_wgrad"] * 1e-3) / 1e12
    coeff_tok_s = rows / (ms["grpo_coeffs"] * 1e-3)
    gb = grpo_bytes(rows, R, False)
    rb = risk_bytes(rows, len(w.units), False)
    key = "qwen2_7b_layer"
    roofs = {
        "compress": roof(key, "compress", comp_b, ms["compress"],
                         what=f"{comp_b} B per call (2 units, row sums on)"),
        "decompress": roof(key, "decompress", decomp_b, ms["decompress"],
                           what=f"{decomp_b} B per call (2 units)"),
        "dequant_wgrad": roof("wgrad_4096", "dequant_wgrad", wflops, ms["dequant_wgrad"],
                              BF16_PEAK_TFLOPS, "TFLOP/s", "mfma", f"{wflops:.0f} FLOP per call"),
        "grpo_coeffs": roof(key, "grpo_coeffs", gb, ms["grpo_coeffs"]),
        "exposure_risk": roof(key, "exposure_risk", rb, ms["exposure_risk"]),
    }
    dominant = max(names, key=lambda n: ms[n])
    graph = {
        "grpo_coeffs": graph_us(lambda i: hl.hilore_grpo_coeffs(
            sets[i]["rewards"], sets[i]["lp_new"], sets[i]["lp_old"], None, None, w.P, w.G, w.T,
            D.CLIP_EPS, D.ADV_EPS, 0.0, 0.0, sets[i]["adv"], sets[i]["ratio"], sets[i]["flags"],
            sets[i]["coeff"]), N_SETS),
        "exposure_risk": graph_us(lambda i: hl.hilore_unit_exposure_risk(
            sets[i]["coeff"], None, rows, sets[i]["uc"], D.EPS_ALPHA, D.EPS_REL, sets[i]["expo"],
            sets[i]["risk"], sets[i]["rel"], workspace=sets[i]["risk_ws"]), N_SETS)}
    out = {
        "metric": METRIC,
        "value": round(codec_gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "qwen2_7b_layer+wgrad_4096",
                   "tokens": rows, "responses": R, "group": w.G,
                   "units": [[u.rows, u.cols] for u in w.units], "code": "fp8-e4m3fn",
                   "block": block, "wgrad_KMN": [K, M, N], "buffer_sets": N_SETS},
        "codec_frac_hbm": round(codec_gbs / HBM_PEAK_GBS, 4),
        "wgrad_tflops": round(wgrad_tflops, 2),
        "wgrad_frac_mfma": round(wgrad_tflops / BF16_PEAK_TFLOPS, 4),
        "coeff_tok_s": round(coeff_tok_s, 1),
        "kernel_us": {n: us_stats(per[k]) for k, n in enumerate(names)},
        "graph_us": graph,
        "roofline": roofs[dominant],
        "rooflines": roofs,
    }
    return out, sets


# ------------------------------------------------------------ other configs --
def tiny_config(args, hl, wl):
    """Latency of the tiny workload: coefficients of 4 x 8 x 32 slots, compress
    (row sums on) and decompress of one 1024x896 activation, int8 1x128."""
    import torch

    w = wl.TINY
    code, block = hl.HILORE_CODE_INT8, w.block
    b = wl.grpo_batch(w.P, w.G, w.T, seed=w.seed)
    rows, cols = w.units[0].rows, w.units[0].cols
    d = {k: torch.from_numpy(getattr(b, k)).cuda() for k in ("rewards", "logp_new", "logp_old")}
    adv = torch.empty(w.P * w.G, device="cuda")
    ratio = torch.empty(rows, device="cuda")
    flags = torch.empty(rows, dtype=torch.uint8, device="cuda")
    coeff = torch.empty(rows, device="cuda")
    x = torch.from_numpy(wl.activation_host(rows, cols, w.seed, outliers=w.outliers)
                         .view("int16")).view(torch.bfloat16).cuda()
    codes = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
    scales = torch.empty((rows, cols // block), device="cuda")
    xhat = torch.empty((rows, cols), dtype=torch.bfloat16, device="cuda")
    ssx = torch.empty(rows, device="cuda")
    sse = torch.empty(rows, device="cuda")
    uc = [hl.unit_desc(x=x, codes=codes, scales=scales, row_ss_x=ssx, row_ss_err=sse)]
    ud = [hl.unit_desc(codes=codes, scales=scales, xhat=xhat)]

    def step(i, mark):
        mark = mark or (lambda k: None)
        mark(0)
        hl.hilore_grpo_coeffs(d["rewards"], d["logp_new"], d["logp_old"], None, None, w.P, w.G,
                              w.T, D.CLIP_EPS, D.ADV_EPS, 0.0, 0.0, adv, ratio, flags, coeff)
        mark(1)
        hl.hilore_compress(uc, code, block)
        mark(2)
        hl.hilore_decompress(ud, code, block)
        mark(3)

    per, _ = timed_steps(step, 3, max(args.steps, 50), args.warmup)
    graph = {
        "grpo_coeffs": graph_us(lambda i: hl.hilore_grpo_coeffs(
            d["rewards"], d["logp_new"], d["logp_old"], None, None, w.P, w.G, w.T, D.CLIP_EPS,
            D.ADV_EPS, 0.0, 0.0, adv, ratio, flags, coeff)),
        "compress": graph_us(lambda i: hl.hilore_compress(uc, code, block)),
        "decompress": graph_us(lambda i: hl.hilore_decompress(ud, code, block))}
    cb, db = codec_bytes(rows, cols, block, stats=True)
    return {"workload": "tiny", "slots": rows, "unit": [rows, cols], "code": "int8", "block": block,
            "latency_us": {"grpo_coeffs": us_stats(per[0]), "compress": us_stats(per[1]),
                           "decompress": us_stats(per[2]),
                           "codec": round((med(per[1]) + med(per[2])) * 1e3, 2)},
            "graph_us": graph,
            "codec_gbs": round((cb + db) / ((med(per[1]) + med(per[2])) * 1e-3) / 1e9, 2),
            "note": "launch-bound: reported as latency (median of per-call HIP events, eager; "
                    "and per call inside a replayed HIP graph)"}


def codec_config(args, hl, wl, key):
    """One step of the codec path over a multi-unit workload, in the order of
    Algorithm 1: coefficients, batched compress with row sums, exposure/risk of
    every L unit, batched decompress.  The working sets (23 GB and 75 GB) are
    far beyond the caches, so one buffer set is used.  Returns the config's
    entry and the host sample of its first unit for the CPU baseline."""
    import numpy as np
    import torch

    w = wl.WORKLOADS[key]
    code = hl.CODES[w.code]
    block = w.block
    if key == "qwen2_7b_plan":
        act = wl.plan_actions(len(w.units), w.seed)
        chosen = [i for i in range(len(w.units)) if act[i] == "L"]
    else:
        chosen = list(range(len(w.units)))
    b = wl.grpo_batch(w.P, w.G, w.T, seed=w.seed, pad_frac=w.pad_frac)
    R = w.P * w.G
    slots = R * w.T
    rows = w.units[0].rows
    assert rows == slots, "coefficients are aligned 1:1 with activation rows"
    progress(f"{key}: drawing {len(chosen)} units of {rows}x{w.units[0].cols} on the device")
    rewards, lp_new, lp_old = (torch.from_numpy(a).cuda() for a in (b.rewards, b.logp_new,
                                                                    b.logp_old))
    mask = torch.from_numpy(b.mask).cuda() if b.mask is not None else None
    adv = torch.empty(R, dtype=torch.float32, device="cuda")
    flags = torch.empty(slots, dtype=torch.uint8, device="cuda")
    coeff = torch.empty(slots, dtype=torch.float32, device="cuda")
    ratio = torch.empty(slots, dtype=torch.float32, device="cuda")
    keep, uc, ud = [], [], []
    for i in chosen:
        u = w.units[i]
        x = wl.activation_device(u.rows, u.cols, w.seed * 1000 + i, dist=w.dist,
                                 outliers=w.outliers)
        codes = torch.empty((u.rows, u.cols), dtype=torch.uint8, device="cuda")
        scales = torch.empty((u.rows, u.cols // block), dtype=torch.float32, device="cuda")
        xhat = torch.empty((u.rows, u.cols), dtype=torch.bfloat16, device="cuda")
        ssx = torch.empty(u.rows, dtype=torch.float32, device="cuda")
        sse = torch.empty(u.rows, dtype=torch.float32, device="cuda")
        keep.append((x, codes, scales, xhat, ssx, sse))
        uc.append(hl.unit_desc(x=x, codes=codes, scales=scales, row_ss_x=ssx, row_ss_err=sse))
        ud.append(hl.unit_desc(codes=codes, scales=scales, xhat=xhat))
    n = len(chosen)
    expo = torch.empty(n, dtype=torch.float32, device="cuda")
    risk = torch.empty(n, dtype=torch.float32, device="cuda")
    rel = torch.empty(n, dtype=torch.float32, device="cuda")
    risk_ws = torch.zeros(hl.hilore_unit_exposure_risk_workspace_bytes(rows, n), dtype=torch.uint8,
                          device="cuda")
    grpo_ws = torch.empty(max(16, hl.hilore_grpo_coeffs_workspace_bytes(w.P, w.G, w.T)),
                          dtype=torch.uint8, device="cuda")
    sample = host_bf16(keep[0][0][:2048])
    torch.cuda.synchronize()
    names = ["grpo_coeffs", "compress", "exposure_risk", "decompress"]

    def step(i, mark):
        mark = mark or (lambda k: None)
        mark(0)
        hl.hilore_grpo_coeffs(rewards, lp_new, lp_old, None, mask, w.P, w.G, w.T, D.CLIP_EPS,
                              D.ADV_EPS, 0.0, 0.0, adv, ratio, flags, coeff, workspace=grpo_ws)
        mark(1)
        hl.hilore_compress(uc, code, block)
        mark(2)
        hl.hilore_unit_exposure_risk(coeff, mask, rows, uc, D.EPS_ALPHA, D.EPS_REL, expo, risk, rel,
                                     workspace=risk_ws)
        mark(3)
        hl.hilore_decompress(ud, code, block)
        mark(4)

    progress(f"{key}: {args.warmup} warm-up and {args.steps} timed steps")
    per, wall = timed_steps(step, len(names), args.steps, args.warmup)
    graph = {
        "grpo_coeffs": graph_us(lambda i: hl.hilore_grpo_coeffs(
            rewards, lp_new, lp_old, None, mask, w.P, w.G, w.T, D.CLIP_EPS, D.ADV_EPS, 0.0, 0.0,
            adv, ratio, flags, coeff, workspace=grpo_ws)),
        "exposure_risk": graph_us(lambda i: hl.hilore_unit_exposure_risk(
            coeff, mask, rows, uc, D.EPS_ALPHA, D.EPS_REL, expo, risk, rel, workspace=risk_ws))}
    ms = {nm: med(per[k]) for k, nm in enumerate(names)}
    comp_b = decomp_b = 0
    for i in chosen:
        c, d = codec_bytes(w.units[i].rows, w.units[i].cols, block, stats=True)
        comp_b += c
        decomp_b += d
    codec_gbs = (comp_b + decomp_b) / ((ms["compress"] + ms["decompress"]) * 1e-3) / 1e9
    masked = mask is not None
    valid = int(b.mask.sum()) if masked else slots
    out = {
        "workload": key, "units": [n, rows, w.units[0].cols], "code": w.code, "block": block,
        "tokens": slots, "valid_tokens": valid, "responses": R, "group": w.G,
        "padded_frac": None if b.mask is None else round(1.0 - valid / slots, 4),
        "round_trip_bytes": comp_b + decomp_b,
        "codec_gbs": round(codec_gbs, 2), "codec_frac_hbm": round(codec_gbs / HBM_PEAK_GBS, 4),
        "coeff_tok_s": round(slots / (ms["grpo_coeffs"] * 1e-3), 1),
        "coeff_valid_tok_s": round(valid / (ms["grpo_coeffs"] * 1e-3), 1),
        "ms_per_step": round(wall * 1e3, 4), "steps": args.steps,
        "kernel_us": {nm: us_stats(per[k]) for k, nm in enumerate(names)},
        "graph_us": graph,
        "rooflines": {
            "compress": roof(key, "compress", comp_b, ms["compress"],
                             what=f"{comp_b} B per call ({n} units, row sums on)"),
            "decompress": roof(key, "decompress", decomp_b, ms["decompress"],
                               what=f"{decomp_b} B per call ({n} units)"),
            "exposure_risk": roof(key, "exposure_risk", risk_bytes(rows, n, masked),
                                  ms["exposure_risk"]),
            "grpo_coeffs": roof(key, "grpo_coeffs", grpo_bytes(slots, R, masked),
                                ms["grpo_coeffs"]),
        },
    }
    del keep, uc, ud
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out, sample


def coeff_calls(args, hl, wl, P, G, T, pad, seed, key, n_norm=0.0, device_draw=False):
    """Median per-call duration of hilore_grpo_coeffs on one batch shape,
    rotating over input sets unless the working set exceeds 1 GB."""
    import torch

    R, n = P * G, P * G * T
    work = n * (18 if pad is not None else 17)
    n_sets = 1 if work > (1 << 30) else N_SETS
    sets = []
    for s in range(n_sets):
        if device_draw:
            rewards, ln, lo, mask = wl.grpo_batch_device(P, G, T, seed + s, pad_frac=pad)
        else:
            b = wl.grpo_batch(P, G, T, seed=seed + s, pad_frac=pad)
            rewards, ln, lo = (torch.from_numpy(a).cuda() for a in (b.rewards, b.logp_new,
                                                                    b.logp_old))
            mask = torch.from_numpy(b.mask).cuda() if b.mask is not None else None
        sets.append({"rewards": rewards, "ln": ln, "lo": lo, "mask": mask,
                     "adv": torch.empty(R, device="cuda"), "ratio": torch.empty(n, device="cuda"),
                     "flags": torch.empty(n, dtype=torch.uint8, device="cuda"),
                     "coeff": torch.empty(n, device="cuda")})
    ws = torch.empty(max(16, hl.hilore_grpo_coeffs_workspace_bytes(P, G, T)), dtype=torch.uint8,
                     device="cuda")
    valid = int(sets[0]["mask"].sum().item()) if sets[0]["mask"] is not None else n

    def step(i, mark):
        st = sets[i]
        mark = mark or (lambda k: None)
        mark(0)
        hl.hilore_grpo_coeffs(st["rewards"], st["ln"], st["lo"], None, st["mask"], P, G, T,
                              D.CLIP_EPS, D.ADV_EPS, 0.0, n_norm, st["adv"], st["ratio"],
                              st["flags"], st["coeff"], workspace=ws)
        mark(1)

    per, _ = timed_steps(step, 1, max(args.steps, 20), args.warmup, n_sets)
    ms = med(per[0])
    g_us = graph_us(lambda i: step(i, None), n_sets)
    gb = grpo_bytes(n, R, pad is not None)
    r = {"P": P, "G": G, "T": T, "slots": n, "valid_tokens": valid,
         "n_norm": "counted" if n_norm <= 0 else "given", "buffer_sets": n_sets,
         "us": us_stats(per[0]), "tok_s": round(n / (ms * 1e-3), 1),
         "valid_tok_s": round(valid / (ms * 1e-3), 1), "graph_us": g_us,
         "graph_tok_s": round(n / (g_us * 1e-6), 1),
         "graph_valid_tok_s": round(valid / (g_us * 1e-6), 1),
         "roofline": roof(key, "grpo_coeffs", gb, ms,
                          what=f"{gb} B per call: 18 B per slot, 8 B per response")}
    del sets
    return r


def coeff_sweep(args, hl, wl):
    """GRPO coefficients on 2^20 .. 2^26 masked slots (G = 16, T = 1024, 30%
    padded, N counted by the pre-pass), inputs drawn on the device; at the
    largest size also with N given (no count)."""
    import torch

    out = []
    for lg in range(20, args.sweep_max_log2 + 1, 2):
        n = 1 << lg
        P = n // (SWEEP_G * SWEEP_T)
        progress(f"coefficient sweep: 2^{lg} slots")
        out.append(coeff_calls(args, hl, wl, P, SWEEP_G, SWEEP_T, SWEEP_PAD, 9000 + lg,
                               f"coeff_sweep_2^{lg}", device_draw=True))
        torch.cuda.empty_cache()
    lg = args.sweep_max_log2
    n = 1 << lg
    out.append(coeff_calls(args, hl, wl, n // (SWEEP_G * SWEEP_T), SWEEP_G, SWEEP_T, SWEEP_PAD,
                           9000 + lg, f"coeff_sweep_2^{lg}_given", n_norm=float(0.7 * n),
                           device_draw=True))
    torch.cuda.empty_cache()
    return out


# -------------------------------------------------------------- context calls --
def alloc_bench(hl, wl, iters=10):
    """Context: hilore_allocate on the profiled plan of a Qwen2-7B-width model
    (28 layers x 7 saved activations of a 16384-token microbatch = 196 units)
    on the paper's 1025 x 1025 grid; per-unit inputs already on the device."""
    import numpy as np
    import torch

    inst = wl.alloc_instance(wl.qwen2_7b_unit_mix(), seed=wl.BASE_SEED + 3)
    n_b, n_d = D.N_B, D.N_DELTA
    d = [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in inst.arrays()]
    action = torch.empty(inst.U, dtype=torch.uint8, device="cuda")
    totals = torch.empty(3, dtype=torch.float64, device="cuda")
    jk = torch.empty(2, dtype=torch.int64, device="cuda")
    ws = torch.empty(hl.hilore_allocate_workspace_bytes(inst.U, n_b, n_d), dtype=torch.uint8,
                     device="cuda")

    def step(i, mark):
        mark = mark or (lambda k: None)
        mark(0)
        hl.hilore_allocate(*d, inst.m_res, inst.delta_b, n_b, n_d, action, totals, jk, ws)
        mark(1)

    per, _ = timed_steps(step, 1, iters, 2)
    ms = med(per[0])
    a = action.cpu().numpy()
    cells = (n_d + 1) * ((n_b + 1 + 63) // 64 * 64)
    # one DP launch per pair of units: read the table before the pair, write the
    # one after it, 2-bit records of both units
    per_pair = cells * 16 + 2 * (cells // 4)
    achieved = per_pair * (inst.U / 2) / (ms * 1e-3) / 1e9
    return {"units": inst.U, "grid": [n_b + 1, n_d + 1], "ms": round(ms, 4),
            "us_per_unit": round(ms * 1e3 / inst.U, 3),
            "table_bytes_per_pair": per_pair,
            "roofline": {"kernel": "allocate_dp", "bound": "hbm", "achieved": round(achieved, 2),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(achieved / HBM_PEAK_GBS, 4),
                         "traffic": TRAFFIC.get("alloc_196/allocate_dp"),
                         "algorithmic": f"{per_pair} B per DP launch (a pair of units); achieved "
                                        "over the whole call, launches and backtrack included"},
            "chosen": {"R": int((a == 0).sum()), "H": int((a == 1).sum()),
                       "L": int((a == 2).sum())}}


def next_rows_bench(args, hl, wl, sets, code, block, rows, R):
    """Context, outside the step: the calls that follow the five hot-path rows,
    on the layer's data.
      lora_grad        hilore_dequant_lora_grad on the MLP unit's codes (16384 x 18944,
                       rank 16): the adapter gradient of the paper's LoRA setting
      grad_rel_err     hilore_grad_rel_err on two 4096 x 4096 fp32 gradients
      calibrate        hilore_calibrate over 8 calibration microbatches x 196 units
      risk_score       hilore_risk_score for 196 units
      update_sparsity  hilore_update_sparsity on the 16384 coefficient slots
      swiglu_bwd       hilore_dequant_swiglu_bwd with the MLP unit's codes as the gate
    Each timed like the step (median of per-call events), rotating over the
    buffer sets."""
    import numpy as np
    import torch

    key = "qwen2_7b_layer_next"  # the profiles' name for these calls on the layer's data

    def timed(fn, iters=20):
        def step(i, mark):
            mark = mark or (lambda k: None)
            mark(0)
            fn(i)
            mark(1)
        per, _ = timed_steps(step, 1, iters, 3, N_SETS)
        return med(per[0])

    out = {}
    w = wl.QWEN2_7B_LAYER
    u = w.units[1]
    K, M, r = u.rows, u.cols, D.LORA_RANK
    dhs = [wl.normal_bf16_device(K, r, 500 + i, 0.05) for i in range(len(sets))]
    da = torch.empty((r, M), dtype=torch.float32, device="cuda")
    ws = torch.empty(hl.hilore_lora_grad_workspace_bytes(K, M, r), dtype=torch.uint8,
                     device="cuda")

    def lora(i):
        _, codes, scales, _, _, _ = sets[i]["keep"][1]
        hl.hilore_dequant_lora_grad(codes, scales, code, block, dhs[i], da, K, M, r,
                                    D.LORA_SCALE, False, ws)

    ms = timed(lora)
    lb = K * M + K * M * 4 // block + K * r * 2 + r * M * 4
    out["lora_grad"] = roof(key, "dequant_lora_grad", lb, ms,
                            what=f"{lb} B per call: codes + scales of {K}x{M}, dh {K}x{r} bf16, "
                                 f"dA {r}x{M} fp32")
    out["lora_grad"]["shape"] = {"K": K, "M": M, "r": r, "code": "fp8-e4m3fn", "block": block}
    # the five rank-16 adapters that share one input (q, k, v or gate, up) in one call
    r5 = 5 * r
    dh5 = [wl.normal_bf16_device(K, r5, 520 + i, 0.05) for i in range(len(sets))]
    da5 = torch.empty((r5, M), dtype=torch.float32, device="cuda")
    ws5 = torch.empty(hl.hilore_lora_grad_workspace_bytes(K, M, r5), dtype=torch.uint8,
                      device="cuda")

    def lora5(i):
        _, codes, scales, _, _, _ = sets[i]["keep"][1]
        hl.hilore_dequant_lora_grad(codes, scales, code, block, dh5[i], da5, K, M, r5,
                                    D.LORA_SCALE, False, ws5)

    ms5 = timed(lora5)
    lb5 = K * M + K * M * 4 // block + K * r5 * 2 + r5 * M * 4
    out["lora_grad_5_adapters"] = {
        "us": round(ms5 * 1e3, 2), "shape": {"K": K, "M": M, "r": r5},
        "achieved_gbs": round(lb5 / (ms5 * 1e-3) / 1e9, 1),
        "vs_one_adapter": round(ms5 / ms, 3),
        "traffic": TRAFFIC.get(f"{key}/dequant_lora_grad_5"),
        "what": f"{r5} adapter rows (five rank-{r} adapters on one input) in one pass over the codes"}
    del dh5, da5, ws5
    n = sets[0]["dw"].numel()
    y = torch.empty(1, dtype=torch.float32, device="cuda")
    wsr = torch.empty(hl.hilore_grad_rel_err_workspace_bytes(n), dtype=torch.uint8, device="cuda")

    def rel(i):
        hl.hilore_grad_rel_err(sets[i]["dw"], sets[(i + 1) % len(sets)]["dw"], y, wsr)

    ms = timed(rel)
    out["grad_rel_err"] = roof(key, "grad_rel_err", 8 * n, ms,
                               what=f"{8 * n} B per call (two fp32 [{n}])")
    nu, nb, nc = 196, 8, 28 * 2
    g = wl.rng(wl.BASE_SEED + 7, 1)
    cls = torch.from_numpy((np.arange(nu) // 7 * 2 + (np.arange(nu) % 7 >= 4)).astype(np.int32)).cuda()
    e = torch.from_numpy(g.uniform(0.1, 2.0, (nb, nu)).astype(np.float32)).cuda()
    rl = torch.from_numpy(g.uniform(1e-3, 5e-2, (nb, nu)).astype(np.float32)).cuda()
    yy = torch.from_numpy(g.uniform(0.0, 1e-2, (nb, nu)).astype(np.float32)).cuda()
    kappa = torch.empty(nc, dtype=torch.float64, device="cuda")
    ebar = torch.empty(nu, dtype=torch.float64, device="cuda")
    psi = torch.empty(nu, dtype=torch.float64, device="cuda")
    out["calibrate_us"] = round(timed(lambda i: hl.hilore_calibrate(cls, e, rl, yy, nc, kappa,
                                                                    ebar)) * 1e3, 2)
    out["risk_score_us"] = round(timed(lambda i: hl.hilore_risk_score(cls, kappa, ebar, e[0],
                                                                      psi)) * 1e3, 2)
    counts = torch.empty(3, dtype=torch.int64, device="cuda")
    share = torch.empty(1, dtype=torch.float64, device="cuda")

    def sparsity(i):
        st = sets[i]
        hl.hilore_update_sparsity(st["coeff"], st["flags"], st["adv"], None, R, rows // R,
                                  D.TOP_FRAC, counts, share)

    out["update_sparsity_us"] = round(timed(sparsity) * 1e3, 2)
    dh2 = wl.normal_bf16_device(K, M, 600, 0.01)
    dg = torch.empty((K, M), dtype=torch.bfloat16, device="cuda")
    du = torch.empty_like(dg)

    def swiglu(i):
        x, codes, scales, _, _, _ = sets[i]["keep"][1]
        hl.hilore_dequant_swiglu_bwd(hl.unit_desc(codes=codes, scales=scales, rows=K, cols=M),
                                     hl.unit_desc(x=x), code, block, dh2, dg, du)

    ms = timed(swiglu)
    sb = K * M * (1 + 2 + 2 + 4) + K * M * 4 // block
    out["swiglu_bwd"] = roof(key, "dequant_swiglu_bwd", sb, ms,
                             what=f"{sb} B per call: gate codes + scales, up and dh bf16, dgate "
                                  f"and dup bf16, {K}x{M}")
    del dh2, dg, du
    return out


def blas_ref(st, code, block, K, M, N, iters=10):
    """Context only: the library GEMM (torch.mm -> hipBLASLt, bf16 in, bf16
    out, fp32 accumulation) on X reconstructed by hilore_decompress, with X^T
    as a transposed view (the layout the fused kernel reads) and after making
    it contiguous.  Not part of the hot path."""
    import torch
    from paper_2609_33570_amd import hilore as hl

    xhat = torch.empty((K, M), dtype=torch.bfloat16, device="cuda")
    hl.hilore_decompress([hl.unit_desc(codes=st["wc"], scales=st["ws"], xhat=xhat)], code, block)
    xt = xhat.t().contiguous()
    res = {}
    for name, a in (("xhatT_view", xhat.t()), ("xhatT_contiguous", xt)):
        for _ in range(3):
            torch.mm(a, st["dy"])
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            torch.mm(a, st["dy"])
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / iters
        res[f"tflops_{name}"] = round(2.0 * K * M * N / (ms * 1e-3) / 1e12, 2)
    res["what"] = "torch.mm bf16 on the reconstructed X (hipBLASLt), same K, M, N; context, not a target"
    return res


# --------------------------------------------------------------- CPU baseline --
def host_info():
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = None
    return {"cpu": model, "logical_cpus": os.cpu_count(), "cpus_available": affinity}


def cpu_samples(sets, layer_block):
    """Host copies (byte for byte) of what the oracle is timed on, taken while
    the layer's buffers are still on the device."""
    st = sets[0]
    K = st["wc"].shape[0]
    return {
        "hidden": host_bf16(st["keep"][0][0][:4096]),
        "mlp": host_bf16(st["keep"][1][0][:2048]),
        "grpo": st["grpo_host"],
        "wc": st["wc"][:, :512].cpu().contiguous().numpy(),
        "ws": st["ws"][:, :512 // layer_block].cpu().contiguous().numpy(),
        "dy": host_bf16(st["dy"][:, :512]),
        "K": K,
        "lora_codes": st["keep"][1][1][:, :256].cpu().contiguous().numpy(),
        "lora_scales": st["keep"][1][2][:, :256 // layer_block].cpu().contiguous().numpy(),
    }


def cpu_baseline(hl, wl, smp, plan_sample, stress_sample, runs=3):
    """The oracle (plain single-threaded C, as it stands) timed on this host on
    bounded samples of the same workloads, each the median of `runs` runs (the
    wgrad subtile runs once and is extrapolated by FLOP count)."""
    import numpy as np

    import oracle

    oracle.lib()

    def timed(fn, n=runs):
        ts = []
        for _ in range(n):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return med(ts)

    def codec(xs, code, block):
        total = 0
        for x in xs:
            cb, db = codec_bytes(x.shape[0], x.shape[1], block, stats=True)
            total += cb + db

        def run():
            for x in xs:
                c, s = oracle.quantize(x, code, block)
                xh = oracle.dequantize(c, s, code, block)
                oracle.row_stats(x, xh)
        dt = timed(run)
        return round(total / dt / 1e9, 4), dt

    e4m3, i8 = hl.HILORE_CODE_FP8_E4M3FN, hl.HILORE_CODE_INT8
    layer_gbs, layer_dt = codec([smp["hidden"], smp["mlp"]], e4m3, 128)
    b = smp["grpo"]
    dt_grpo = timed(lambda: oracle.grpo_coeffs(b.rewards, b.logp_new, b.logp_old, None, None,
                                               b.P, b.G, b.T))
    # tiny workload in full
    tw = wl.TINY
    tb = wl.grpo_batch(tw.P, tw.G, tw.T, seed=tw.seed)
    tx = wl.activation_host(1024, 896, tw.seed, outliers=tw.outliers)
    dt_tg = timed(lambda: oracle.grpo_coeffs(tb.rewards, tb.logp_new, tb.logp_old, None, None,
                                             tw.P, tw.G, tw.T))
    tiny_gbs, dt_tc = codec([tx], i8, 128)
    plan_gbs, plan_dt = codec([plan_sample], i8, 64)
    stress_gbs, stress_dt = codec([stress_sample], i8, 128)
    sw = wl.LLAMA3_8B_STRESS
    sb = wl.grpo_batch(sw.P, sw.G, sw.T, seed=sw.seed, pad_frac=sw.pad_frac)
    dt_sg = timed(lambda: oracle.grpo_coeffs(sb.rewards, sb.logp_new, sb.logp_old, None, sb.mask,
                                             sw.P, sw.G, sw.T))
    # wgrad: the 512 x 512 x 16384 fp64 subtile, once, extrapolated by FLOP count
    K = smp["K"]
    t0 = time.perf_counter()
    oracle.wgrad(smp["wc"], smp["ws"], e4m3, 128, smp["dy"], variant=0)
    dt_w = time.perf_counter() - t0
    sub_tflops = 2.0 * K * 512 * 512 / dt_w / 1e12
    inst = wl.alloc_instance(wl.qwen2_7b_unit_mix(), seed=wl.BASE_SEED + 3)
    dt_alloc = timed(lambda: oracle.allocate(*inst.arrays(), inst.m_res, inst.delta_b,
                                             n_b=D.N_B, n_d=D.N_DELTA))
    lc, lsc = smp["lora_codes"], smp["lora_scales"]
    dh = wl.normal_bf16_host(lc.shape[0], 16, seed=wl.BASE_SEED + 9, sigma=0.05)
    dt_lora = timed(lambda: oracle.lora_down_grad(lc, lsc, e4m3, 128, dh, scale=D.LORA_SCALE,
                                                  variant=0))
    lora_bytes = lc.size + lsc.size * 4 + dh.size * 2 + 16 * 256 * 4
    return {
        "value": layer_gbs,
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"compress (row sums on) + decompress of the first {smp['hidden'].shape[0]} rows "
                  f"of the 16384x3584 hidden unit and {smp['mlp'].shape[0]} rows of the "
                  f"16384x18944 MLP unit (fp8-e4m3 1x128); median of {runs} runs of "
                  f"{layer_dt:.2f} s",
        "statistic": f"median of {runs} runs (wgrad subtile: one run)",
        "host": host_info(),
        "threads_used": 1,
        "configs": {
            "tiny": {"coeff_us": round(dt_tg * 1e6, 1), "codec_us": round(dt_tc * 1e6, 1),
                     "codec_gbs": tiny_gbs, "sample": "the whole workload"},
            "qwen2_7b_layer": {"codec_gbs": layer_gbs,
                               "coeff_tok_s": round(b.P * b.G * b.T / dt_grpo, 1),
                               "sample": "codec: the rows above; coefficients: all 16384 slots"},
            "qwen2_7b_plan": {"codec_gbs": plan_gbs,
                              "sample": f"compress + decompress of {plan_sample.shape[0]} rows "
                                        f"of one 16384x3584 unit, int8 1x64 ({plan_dt:.2f} s)"},
            "wgrad_4096": {"tflops_extrapolated": round(sub_tflops, 6),
                           "subtile_s": round(dt_w, 2),
                           "sample": f"dW[0:512, 0:512] over K={K} in fp64 (one run), "
                                     "extrapolated to 4096x4096 by FLOP count: "
                                     f"{dt_w * 64:.0f} s for the full dW"},
            "llama3_8b_stress": {"codec_gbs": stress_gbs,
                                 "coeff_tok_s": round(sw.P * sw.G * sw.T / dt_sg, 1),
                                 "sample": f"compress + decompress of {stress_sample.shape[0]} "
                                           f"rows of one 32768x14336 unit, int8 1x128 "
                                           f"({stress_dt:.2f} s); coefficients: all 32768 "
                                           "slots"},
        },
        "allocate_ms": round(dt_alloc * 1e3, 1),
        "allocate_sample": "the same 196-unit plan on the 1025 x 1025 grid",
        "lora_grad_gbs": round(lora_bytes / dt_lora / 1e9, 4),
        "lora_grad_sample": f"rank-16 dA over {lc.shape[0]}x256 MLP codes in fp64",
    }


def wgrad_standalone(hl, sets, code, block, K, M, N, iters=20):
    """The fused wgrad call of the step timed back to back over the rotating
    buffer sets (median of per-call events), outside the step: the kernel's
    own rate, without the decompress that precedes it in the step."""
    import torch

    def call(i):
        st = sets[i % len(sets)]
        hl.hilore_dequant_wgrad(st["wc"], st["ws"], code, block, st["dy"], st["dw"], K, M, N,
                                False)

    for i in range(3):
        call(i)
    torch.cuda.synchronize()
    ts = []
    for i in range(iters):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        call(i)
        e1.record()
        e1.synchronize()
        ts.append(e0.elapsed_time(e1))
    ms = med(ts)
    tf = 2.0 * K * M * N / (ms * 1e-3) / 1e12
    return {"tflops": round(tf, 2), "frac_mfma": round(tf / BF16_PEAK_TFLOPS, 4),
            "us": round(ms * 1e3, 2),
            "what": f"the same call back to back over the {len(sets)} rotating buffer sets "
                    f"({iters} calls, median), outside the step"}


def copy_peak():
    """The streaming rate this GPU reaches with a plain copy of 1 GiB (1 GiB read
    and 1 GiB written, median of 10), which each HBM-bound roofline is also read
    against ("frac_copy"): torch's elementwise kernel (x * 1.0 in bf16, an exact
    copy) and, for reference, the runtime's device-to-device blit (copy_)."""
    import torch
    n = 1 << 29  # bf16 elements: 1 GiB
    src = torch.ones(n, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)

    def rate(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(10):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1))
        return 2 * 2 * n / (med(ts) * 1e-3) / 1e9

    elementwise = rate(lambda: torch.mul(src, 1.0, out=dst))
    blit = rate(lambda: dst.copy_(src))
    del src, dst
    torch.cuda.empty_cache()
    return {"gbs": round(elementwise, 1), "frac_of_peak": round(elementwise / HBM_PEAK_GBS, 4),
            "blit_gbs": round(blit, 1),
            "what": "1 GiB bf16 copied by torch's elementwise kernel (x * 1.0), 1 GiB read + "
                    "1 GiB written, median of 10; blit_gbs: the runtime's device-to-device copy_"}


def add_copy_fractions(o, copy_gbs):
    """Add achieved / copy peak next to every HBM-bound roofline in the line."""
    if isinstance(o, dict):
        if o.get("bound") == "hbm" and isinstance(o.get("achieved"), (int, float)):
            o["frac_copy"] = round(o["achieved"] / copy_gbs, 4)
        for v in o.values():
            add_copy_fractions(v, copy_gbs)
    elif isinstance(o, list):
        for v in o:
            add_copy_fractions(v, copy_gbs)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the hot path shards without communication except one dW reduce-scatter, "
              "which this library does not implement)", file=sys.stderr)
        return 2

    import torch

    from paper_2609_33570_amd import hilore as hl
    from paper_2609_33570_amd import workloads as wl

    hl.load()
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    TRAFFIC.update(measured_traffic())

    out, sets = layer_step(args, hl, wl)
    ww = wl.WGRAD_4096
    code, block = hl.HILORE_CODE_FP8_E4M3FN, 128
    if not args.step_only:
        w = wl.QWEN2_7B_LAYER
        R = w.P * w.G
        progress("context calls: the H/L/R allocation of a 196-unit plan")
        out["allocate"] = alloc_bench(hl, wl)
        progress("context calls: LoRA adapter gradient, calibration and diagnostics")
        out["next"] = next_rows_bench(args, hl, wl, sets, code, block, R * w.T, R)
    wg_alone = None
    if not args.step_only:
        progress("the fused wgrad back to back, outside the step")
        wg_alone = wgrad_standalone(hl, sets, code, block, *ww.wgrad)
    if args.blas_ref:
        progress("timing hipBLASLt on the reconstructed X")
        out["blas_ref"] = blas_ref(sets[0], code, block, *ww.wgrad)
    smp = None if args.no_cpu_baseline else cpu_samples(sets, block)
    del sets
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    plan_sample = stress_sample = None
    if not args.step_only:
        k = out["kernel_us"]
        out["configs"] = {
            "tiny": tiny_config(args, hl, wl),
            "qwen2_7b_layer": {"workload": "qwen2_7b_layer", "codec_gbs": out["value"],
                               "codec_frac_hbm": out["codec_frac_hbm"],
                               "coeff_tok_s": out["coeff_tok_s"],
                               "exposure_risk_us": k["exposure_risk"],
                               "see": "the headline step"},
            "wgrad_4096": {"workload": "wgrad_4096", "tflops": out["wgrad_tflops"],
                           "frac_mfma": out["wgrad_frac_mfma"], "KMN": list(ww.wgrad),
                           "see": "the headline step", "standalone": wg_alone},
        }
        out["configs"]["qwen2_7b_plan"], plan_sample = codec_config(args, hl, wl, "qwen2_7b_plan")
        stress, stress_sample = codec_config(args, hl, wl, "llama3_8b_stress")
        sw = wl.LLAMA3_8B_STRESS
        progress("llama3_8b_stress: coefficients at 32768 and 65536 slots")
        stress["coeff_calls"] = [
            coeff_calls(args, hl, wl, sw.P, sw.G, T, sw.pad_frac, sw.seed + 10 * T,
                        f"llama3_8b_stress_T{T}") for T in (sw.T, 2 * sw.T)]
        out["configs"]["llama3_8b_stress"] = stress
        out["coeff_sweep"] = coeff_sweep(args, hl, wl)
    progress("copy peak: 1 GiB device-to-device")
    out["copy_peak"] = copy_peak()
    add_copy_fractions(out, out["copy_peak"]["gbs"])
    if smp is not None:
        progress("timing the oracle on the host")
        if plan_sample is None:
            plan_sample = wl.activation_host(2048, 3584, 7, outliers=("channels", 0.005, 30.0))
            stress_sample = wl.activation_host(1024, 14336, 8, dist="student_t3")
        out["cpu_baseline"] = cpu_baseline(hl, wl, smp, plan_sample[:2048], stress_sample[:1024])
    print(json.dumps(out))
    return 0


if __name__ == "__main__":
    sys.exit(main())
