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
coefficient tokens/s ride along, each with its own roofline.  For context the
line also times hilore_allocate (the H/L/R dynamic programme that follows the
exposure step) on a 196-unit plan, and, under "next", the calls that follow
the five rows (the LoRA adapter gradient and the gated-MLP activation backward
on the MLP unit, the calibration scalars, the update-sparsity diagnostics), all
outside the step.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

from paper_2609_33570_amd import defaults as D

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "compress+decompress GB/s (% HBM peak); fused dequant-wgrad TFLOP/s; coeff tok/s"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
N_SETS = 4


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a plain 1 GiB device copy (for scaling HBM byte counters)")
    p.add_argument("--blas-ref", action="store_true",
                   help="also time hipBLASLt's bf16 GEMM (torch.mm) on the reconstructed X, for context")
    p.add_argument("--cpu-rows", type=int, default=8192,
                   help="MLP rows (and 4x as many hidden rows) in the oracle's timed sample")
    p.add_argument("--workload", default="qwen2_7b_layer",
                   choices=["qwen2_7b_layer", "qwen2_7b_plan", "llama3_8b_stress"],
                   help="qwen2_7b_layer: the full step with the 4096^3 wgrad (default); the "
                        "others time coefficients + compress + exposure/risk + decompress of "
                        "the whole-model plan (78 L units) or the Llama-3-8B-shaped stress case")
    return p.parse_args()


def codec_bytes(rows, cols, block, stats):
    """Algorithmic HBM bytes of one compress and one decompress of a unit:
    read bf16 x, write codes + scales (+ two fp32 row sums); read codes +
    scales, write bf16 xhat."""
    n = rows * cols
    scales = 4 * n // block
    comp = 2 * n + n + scales + (8 * rows if stats else 0)
    decomp = n + scales + 2 * n
    return comp, decomp


def measured_traffic():
    """HBM bytes per launch from the committed rocprofv3 counter summary, for
    the kernels whose sources are unchanged since the counters were taken."""
    import hashlib

    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(path):
        return {}
    table = json.load(open(path))
    csrc = os.path.join(ROOT, "paper_2609_33570_amd", "csrc")
    common = ["device_common.hpp", "hilore_internal.hpp"]
    files = {"compress": ["codec.hip"], "decompress": ["codec.hip"], "dequant_wgrad": ["wgrad.hip"],
             "grpo_coeffs": ["grpo.hip"], "exposure_risk": ["risk.hip"],
             "dequant_lora_grad": ["lora.hip"], "grad_rel_err": ["calib.hip"],
             "dequant_swiglu_bwd": ["swiglu.hip"], "allocate_dp": ["alloc.hip"]}
    out = {}
    for k, ent in table.get("kernels", {}).items():
        h = hashlib.sha256()
        for f in files.get(k, []) + common:
            with open(os.path.join(csrc, f), "rb") as fh:
                h.update(fh.read())
        out[k] = ent["traffic_bytes"] if h.hexdigest() == ent["source_sha256"] else None
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the hot path shards without communication except one dW reduce-scatter, "
              "which this library does not implement)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2609_33570_amd import hilore as hl
    from paper_2609_33570_amd import workloads as wl

    hl.load()
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    torch.cuda.set_device(0)
    if args.workload != "qwen2_7b_layer":
        return codec_workload(args, hl, wl)

    w = wl.QWEN2_7B_LAYER
    ww = wl.WGRAD_4096
    code, block = hl.HILORE_CODE_FP8_E4M3FN, 128
    K, M, N = ww.wgrad
    R = w.P * w.G
    rows = R * w.T
    b = wl.grpo_batch(w.P, w.G, w.T, seed=w.seed)

    def progress(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    # ---------------------------------------------------------------- setup --
    progress("drawing inputs on the device")
    sets = []
    for s in range(N_SETS):
        st = {}
        st["grpo_host"] = b
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
        st["risk_ws"] = torch.empty(hl.hilore_unit_exposure_risk_workspace_bytes(rows, len(w.units)),
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

    def step(st, ev=None):
        def mark(i):
            if ev is not None:
                ev[i].record()
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
    progress("warm-up")
    for i in range(args.warmup):
        step(sets[i % N_SETS])
    torch.cuda.synchronize()
    progress(f"timing {args.steps} steps")

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(sets[i % N_SETS], events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    per = {n: [] for n in names}
    for ev in events:
        for k, n in enumerate(names):
            per[n].append(ev[k].elapsed_time(ev[k + 1]))
    avg = {n: float(np.mean(v)) for n, v in per.items()}  # ms

    comp_b = decomp_b = 0
    for u in w.units:
        c, d = codec_bytes(u.rows, u.cols, block, stats=True)
        comp_b += c
        decomp_b += d
    codec_gbs = (comp_b + decomp_b) / ((avg["compress"] + avg["decompress"]) * 1e-3) / 1e9
    wflops = 2.0 * K * M * N
    wgrad_tflops = wflops / (avg["dequant_wgrad"] * 1e-3) / 1e12
    coeff_tok_s = rows / (avg["grpo_coeffs"] * 1e-3)
    grpo_bytes = rows * (4 + 4 + 4 + 4 + 1) + R * 8
    risk_bytes = rows * (4 + 4) * len(w.units) + rows * 4

    traffic = measured_traffic()

    def roof(name, achieved, peak, unit, bound, per_unit):
        return {"kernel": name, "bound": bound, "achieved": round(achieved, 2), "peak": peak,
                "unit": unit, "frac": round(achieved / peak, 4), "traffic": traffic.get(name),
                "algorithmic": per_unit}

    roofs = {
        "compress": roof("compress", comp_b / (avg["compress"] * 1e-3) / 1e9, HBM_PEAK_GBS,
                         "GB/s", "hbm", f"{comp_b} B per launch (2 units)"),
        "decompress": roof("decompress", decomp_b / (avg["decompress"] * 1e-3) / 1e9,
                           HBM_PEAK_GBS, "GB/s", "hbm", f"{decomp_b} B per launch (2 units)"),
        "dequant_wgrad": roof("dequant_wgrad", wgrad_tflops, BF16_PEAK_TFLOPS, "TFLOP/s", "mfma",
                              f"{wflops:.0f} FLOP per launch"),
        "grpo_coeffs": roof("grpo_coeffs", grpo_bytes / (avg["grpo_coeffs"] * 1e-3) / 1e9,
                            HBM_PEAK_GBS, "GB/s", "hbm", f"{grpo_bytes} B per launch"),
        "exposure_risk": roof("exposure_risk", risk_bytes / (avg["exposure_risk"] * 1e-3) / 1e9,
                              HBM_PEAK_GBS, "GB/s", "hbm", f"{risk_bytes} B per launch"),
    }
    dominant = max(names, key=lambda n: avg[n])

    out = {
        "metric": METRIC,
        "value": round(codec_gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4),
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
        "kernel_ms": {n: round(v, 5) for n, v in avg.items()},
        "roofline": roofs[dominant],
        "rooflines": roofs,
    }

    progress("timing the H/L/R allocation of a 196-unit plan")
    out["allocate"] = alloc_bench(hl, wl)
    progress("timing the LoRA adapter gradient, calibration and diagnostics")
    out["next"] = next_rows_bench(hl, wl, sets, w, code, block, rows, R)
    if args.blas_ref:
        progress("timing hipBLASLt on the reconstructed X")
        out["blas_ref"] = blas_ref(sets[0], code, block, K, M, N)
    if not args.no_cpu_baseline:
        progress("timing the oracle on the host")
        out["cpu_baseline"] = cpu_baseline(args, sets[0], w, block, code)
    print(json.dumps(out))
    return 0


def codec_workload(args, hl, wl):
    """One step of the codec path over a multi-unit workload, in the order of
    Algorithm 1: coefficients, batched compress with row sums, exposure/risk
    of every L unit, batched decompress.  The working sets (23 GB and 75 GB)
    are far beyond the caches, so no buffer rotation is needed."""
    import numpy as np
    import torch

    import oracle  # noqa: F401  (imported for the CPU baseline only)

    w = wl.WORKLOADS[args.workload]
    code = hl.CODES[w.code]
    block = w.block
    if w.key == "qwen2_7b_plan":
        act = wl.plan_actions(len(w.units), w.seed)
        chosen = [i for i in range(len(w.units)) if act[i] == "L"]
    else:
        chosen = list(range(len(w.units)))
    b = wl.grpo_batch(w.P, w.G, w.T, seed=w.seed, pad_frac=w.pad_frac)
    R = w.P * w.G
    slots = R * w.T
    rows = w.units[0].rows
    assert rows == slots, "coefficients are aligned 1:1 with activation rows"

    def progress(msg):
        print(f"[bench] {msg}", file=sys.stderr, flush=True)

    progress(f"drawing {len(chosen)} units of {rows}x{w.units[0].cols} on the device")
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
    risk_ws = torch.empty(hl.hilore_unit_exposure_risk_workspace_bytes(rows, n), dtype=torch.uint8,
                          device="cuda")
    grpo_ws = torch.empty(max(16, hl.hilore_grpo_coeffs_workspace_bytes(w.P, w.G, w.T)),
                          dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    names = ["grpo_coeffs", "compress", "exposure_risk", "decompress"]

    def step(ev=None):
        def mark(i):
            if ev is not None:
                ev[i].record()
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

    steps = min(args.steps, 5)
    progress("warm-up")
    for _ in range(max(1, min(args.warmup, 2))):
        step()
    torch.cuda.synchronize()
    progress(f"timing {steps} steps")
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        step(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    avg = {nm: float(np.mean([ev[k].elapsed_time(ev[k + 1]) for ev in events]))
           for k, nm in enumerate(names)}
    comp_b = decomp_b = 0
    for i in chosen:
        c, d = codec_bytes(w.units[i].rows, w.units[i].cols, block, stats=True)
        comp_b += c
        decomp_b += d
    codec_gbs = (comp_b + decomp_b) / ((avg["compress"] + avg["decompress"]) * 1e-3) / 1e9
    grpo_bytes = slots * (4 + 4 + 4 + 4 + 1 + (1 if mask is not None else 0)) + R * 8
    risk_bytes = rows * (4 + 4) * n + rows * (4 + (1 if mask is not None else 0))

    def roof(name, nbytes):
        a = nbytes / (avg[name] * 1e-3) / 1e9
        return {"kernel": name, "bound": "hbm", "achieved": round(a, 2), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(a / HBM_PEAK_GBS, 4), "traffic": None,
                "algorithmic": f"{nbytes} B per launch"}

    roofs = {"compress": roof("compress", comp_b), "decompress": roof("decompress", decomp_b),
             "grpo_coeffs": roof("grpo_coeffs", grpo_bytes),
             "exposure_risk": roof("exposure_risk", risk_bytes)}
    dominant = max(names, key=lambda k: avg[k])
    out = {
        "metric": METRIC, "value": round(codec_gbs, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": steps, "warmup": max(1, min(args.warmup, 2)),
        "ms_per_step": round(wall / steps * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.key, "tokens": slots, "responses": R, "group": w.G,
                   "units": [len(chosen), rows, w.units[0].cols], "code": w.code,
                   "block": block, "padded_frac": None if b.mask is None else
                   round(1.0 - float(b.mask.mean()), 4)},
        "codec_frac_hbm": round(codec_gbs / HBM_PEAK_GBS, 4),
        "coeff_tok_s": round(slots / (avg["grpo_coeffs"] * 1e-3), 1),
        "kernel_ms": {k: round(v, 5) for k, v in avg.items()},
        "roofline": roofs[dominant], "rooflines": roofs,
    }
    if not args.no_cpu_baseline:
        progress("timing the oracle on the host")
        import oracle

        oracle.lib()
        n_rows = min(rows, 4096)
        x = keep[0][0][:n_rows].cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
        t0 = time.perf_counter()
        c, sc = oracle.quantize(x, code, block)
        xh = oracle.dequantize(c, sc, code, block)
        oracle.row_stats(x, xh)
        dt = time.perf_counter() - t0
        cb, db = codec_bytes(n_rows, x.shape[1], block, stats=True)
        out["cpu_baseline"] = {"value": round((cb + db) / dt / 1e9, 4), "unit": "GB/s",
                               "cores": 1, "kind": "oracle",
                               "sample": f"compress+decompress of {n_rows}x{x.shape[1]} rows of "
                                         f"the first unit ({w.code} 1x{block}); {dt:.1f} s"}
    print(json.dumps(out))
    return 0


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

    def call():
        hl.hilore_allocate(*d, inst.m_res, inst.delta_b, n_b, n_d, action, totals, jk, ws)

    for _ in range(2):
        call()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(iters):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / iters
    a = action.cpu().numpy()
    cells = (n_b + 1) * ((n_b + 1 + 63) // 64 * 64)
    per_unit = cells * 16 + cells // 4  # read the previous table, write the next, 2-bit records
    achieved = per_unit * inst.U / (ms * 1e-3) / 1e9
    return {"units": inst.U, "grid": [n_b + 1, n_d + 1], "ms": round(ms, 4),
            "us_per_unit": round(ms * 1e3 / inst.U, 3),
            "table_bytes_per_unit": per_unit,
            "roofline": {"kernel": "allocate_dp", "bound": "hbm", "achieved": round(achieved, 2),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(achieved / HBM_PEAK_GBS, 4),
                         "traffic": measured_traffic().get("allocate_dp"),
                         "algorithmic": f"{per_unit} B per unit (one DP launch); achieved over "
                                        "the whole call, launches and backtrack included"},
            "chosen": {"R": int((a == 0).sum()), "H": int((a == 1).sum()),
                       "L": int((a == 2).sum())}}


def next_rows_bench(hl, wl, sets, w, code, block, rows, R, iters=20):
    """Context, outside the step: the calls that follow the five hot-path rows,
    on this microbatch's data.
      lora_grad        hilore_dequant_lora_grad on the MLP unit's codes (16384 x 18944,
                       rank 16): the adapter gradient of the paper's LoRA setting
      grad_rel_err     hilore_grad_rel_err on two 4096 x 4096 fp32 gradients
      calibrate        hilore_calibrate over 8 calibration microbatches x 196 units
      risk_score       hilore_risk_score for 196 units
      update_sparsity  hilore_update_sparsity on the 16384 coefficient slots
      swiglu_bwd       hilore_dequant_swiglu_bwd with the MLP unit's codes as the gate
    Each timed with HIP events on the stream it runs on, averaged over `iters`
    calls that rotate over the buffer sets."""
    import numpy as np
    import torch

    def timed(fn):
        for i in range(3):
            fn(i)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for i in range(iters):
            fn(i)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / iters  # ms

    def roof(name, nbytes, ms, per_unit):
        a = nbytes / (ms * 1e-3) / 1e9
        return {"kernel": name, "bound": "hbm", "achieved": round(a, 2), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(a / HBM_PEAK_GBS, 4), "us": round(ms * 1e3, 2),
                "algorithmic": per_unit}

    out = {}
    # LoRA adapter gradient on the MLP unit of each set
    u = w.units[1]
    K, M, r = u.rows, u.cols, D.LORA_RANK
    dhs = [wl.normal_bf16_device(K, r, 500 + i, 0.05) for i in range(len(sets))]
    da = torch.empty((r, M), dtype=torch.float32, device="cuda")
    ws = torch.empty(hl.hilore_lora_grad_workspace_bytes(K, M, r), dtype=torch.uint8,
                     device="cuda")

    def lora(i):
        st = sets[i % len(sets)]
        _, codes, scales, _, _, _ = st["keep"][1]
        hl.hilore_dequant_lora_grad(codes, scales, code, block, dhs[i % len(sets)], da, K, M, r,
                                    D.LORA_SCALE, False, ws)

    ms = timed(lora)
    lb = K * M + K * M * 4 // block + K * r * 2 + r * M * 4
    out["lora_grad"] = roof("dequant_lora_grad", lb, ms,
                            f"{lb} B per call: codes + scales of {K}x{M}, dh {K}x{r} bf16, "
                            f"dA {r}x{M} fp32")
    out["lora_grad"]["shape"] = {"K": K, "M": M, "r": r, "code": "fp8-e4m3fn", "block": block}
    traffic = measured_traffic()
    out["lora_grad"]["traffic"] = traffic.get("dequant_lora_grad")
    # relative gradient error of two dW-sized fp32 gradients (the step's dW of two sets)
    n = sets[0]["dw"].numel()
    y = torch.empty(1, dtype=torch.float32, device="cuda")
    wsr = torch.empty(hl.hilore_grad_rel_err_workspace_bytes(n), dtype=torch.uint8, device="cuda")

    def rel(i):
        hl.hilore_grad_rel_err(sets[i % len(sets)]["dw"], sets[(i + 1) % len(sets)]["dw"], y, wsr)

    ms = timed(rel)
    out["grad_rel_err"] = roof("grad_rel_err", 8 * n, ms, f"{8 * n} B per call (two fp32 [{n}])")
    out["grad_rel_err"]["traffic"] = traffic.get("grad_rel_err")
    # calibration scalars and risk scores: 196 units (28 layers x 7), 8 calibration microbatches
    nu, nb, nc = 196, 8, 28 * 2
    g = wl.rng(wl.BASE_SEED + 7, 1)
    cls = torch.from_numpy((np.arange(nu) // 7 * 2 + (np.arange(nu) % 7 >= 4)).astype(np.int32)).cuda()
    e = torch.from_numpy(g.uniform(0.1, 2.0, (nb, nu)).astype(np.float32)).cuda()
    rl = torch.from_numpy(g.uniform(1e-3, 5e-2, (nb, nu)).astype(np.float32)).cuda()
    yy = torch.from_numpy(g.uniform(0.0, 1e-2, (nb, nu)).astype(np.float32)).cuda()
    kappa = torch.empty(nc, dtype=torch.float64, device="cuda")
    ebar = torch.empty(nu, dtype=torch.float64, device="cuda")
    psi = torch.empty(nu, dtype=torch.float64, device="cuda")
    ms = timed(lambda i: hl.hilore_calibrate(cls, e, rl, yy, nc, kappa, ebar))
    out["calibrate_us"] = round(ms * 1e3, 2)
    ms = timed(lambda i: hl.hilore_risk_score(cls, kappa, ebar, e[0], psi))
    out["risk_score_us"] = round(ms * 1e3, 2)
    counts = torch.empty(3, dtype=torch.int64, device="cuda")
    share = torch.empty(1, dtype=torch.float64, device="cuda")

    def sparsity(i):
        st = sets[i % len(sets)]
        hl.hilore_update_sparsity(st["coeff"], st["flags"], st["adv"], None, R, rows // R,
                                  D.TOP_FRAC, counts, share)

    ms = timed(sparsity)
    out["update_sparsity_us"] = round(ms * 1e3, 2)
    # gated-MLP activation backward with the gate in L: the MLP unit's codes as g, its
    # bf16 activation as u, a bf16 dh of the same shape
    dh2 = wl.normal_bf16_device(K, M, 600, 0.01)
    dg = torch.empty((K, M), dtype=torch.bfloat16, device="cuda")
    du = torch.empty_like(dg)

    def swiglu(i):
        st = sets[i % len(sets)]
        x, codes, scales, _, _, _ = st["keep"][1]
        hl.hilore_dequant_swiglu_bwd(hl.unit_desc(codes=codes, scales=scales, rows=K, cols=M),
                                     hl.unit_desc(x=x), code, block, dh2, dg, du)

    ms = timed(swiglu)
    sb = K * M * (1 + 2 + 2 + 4) + K * M * 4 // block
    out["swiglu_bwd"] = roof("dequant_swiglu_bwd", sb, ms,
                             f"{sb} B per call: gate codes + scales, up and dh bf16, dgate and dup "
                             f"bf16, {K}x{M}")
    out["swiglu_bwd"]["traffic"] = traffic.get("dequant_swiglu_bwd")
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


def cpu_baseline(args, st, w, block, code):
    """The oracle (plain single-threaded C, as it stands) timed on this host on
    a bounded sample of the same workload: compress (with row sums) and
    decompress of the first --cpu-rows MLP rows and 4x as many hidden rows,
    copied from the device byte for byte; plus the GRPO coefficients of the
    full microbatch and a 128x128 corner of the wgrad, reported alongside."""
    import numpy as np
    import torch

    import oracle

    oracle.lib()
    n_mlp = min(args.cpu_rows, st["keep"][1][0].shape[0])
    n_hid = min(4 * args.cpu_rows, st["keep"][0][0].shape[0])
    xs = [st["keep"][0][0][:n_hid], st["keep"][1][0][:n_mlp]]
    xs = [x.cpu().contiguous().view(torch.int16).numpy().view(np.uint16) for x in xs]
    total = 0
    t0 = time.perf_counter()
    for x in xs:
        c, s = oracle.quantize(x, code, block)
        xh = oracle.dequantize(c, s, code, block)
        oracle.row_stats(x, xh)
        cb, db = codec_bytes(x.shape[0], x.shape[1], block, stats=True)
        total += cb + db
    dt_codec = time.perf_counter() - t0

    b = st["grpo_host"]
    t0 = time.perf_counter()
    oracle.grpo_coeffs(b.rewards, b.logp_new, b.logp_old, None, None, b.P, b.G, b.T)
    dt_grpo = time.perf_counter() - t0

    K = st["wc"].shape[0]
    wc = st["wc"][:, :128].cpu().contiguous().numpy()
    ws = st["ws"][:, :1].cpu().contiguous().numpy()
    dy = st["dy"][:, :128].cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
    t0 = time.perf_counter()
    oracle.wgrad(wc, ws, code, block, dy, variant=0)
    dt_w = time.perf_counter() - t0
    from paper_2609_33570_amd import workloads as wl

    inst = wl.alloc_instance(wl.qwen2_7b_unit_mix(), seed=wl.BASE_SEED + 3)
    t0 = time.perf_counter()
    oracle.allocate(*inst.arrays(), inst.m_res, inst.delta_b, n_b=D.N_B, n_d=D.N_DELTA)
    dt_alloc = time.perf_counter() - t0
    # LoRA adapter gradient (rank 16) on the first 256 columns of the MLP unit
    _, mc, msc, _, _, _ = st["keep"][1]
    lc = mc[:, :256].cpu().contiguous().numpy()
    lsc = msc[:, :256 // block].cpu().contiguous().numpy()
    dh = wl.normal_bf16_host(lc.shape[0], 16, seed=wl.BASE_SEED + 9, sigma=0.05)
    t0 = time.perf_counter()
    oracle.lora_down_grad(lc, lsc, code, block, dh, scale=D.LORA_SCALE, variant=0)
    dt_lora = time.perf_counter() - t0
    lora_bytes = lc.size + lsc.size * 4 + dh.size * 2 + 16 * 256 * 4
    return {
        "value": round(total / dt_codec / 1e9, 4),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"compress+decompress of {n_hid}x{xs[0].shape[1]} hidden and "
                  f"{n_mlp}x{xs[1].shape[1]} MLP rows (fp8-e4m3 1x{block}); "
                  f"{dt_codec:.1f} s",
        "coeff_tok_s": round(b.P * b.G * b.T / dt_grpo, 1),
        "wgrad_tflops": round(2.0 * K * 128 * 128 / dt_w / 1e12, 6),
        "wgrad_sample": f"dW[0:128, 0:128] over K={K} in fp64, {dt_w:.1f} s",
        "allocate_ms": round(dt_alloc * 1e3, 1),
        "allocate_sample": "the same 196-unit plan on the 1025 x 1025 grid",
        "lora_grad_gbs": round(lora_bytes / dt_lora / 1e9, 4),
        "lora_grad_sample": f"rank-16 dA over {lc.shape[0]}x256 MLP codes in fp64, {dt_lora:.1f} s",
    }


if __name__ == "__main__":
    sys.exit(main())
