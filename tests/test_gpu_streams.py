"""The entry points keep no state: two host threads, each on its own stream
(default priority) with its own buffers, run the codec and the weight
gradient repeatedly and concurrently, and every result equals the same call
run alone on the default stream, bit for bit."""
import threading

import pytest
import torch

from paper_2609_33570_amd import workloads as wl
from gpu_util import assert_bytes_equal, host

pytestmark = pytest.mark.gpu

ROWS, COLS, BLOCK, CODE = 4096, 3584, 128, 1  # E4M3FN 1x128
K, M, N = 2048, 1024, 512


def make_job(hl, seed):
    x = wl.activation_device(ROWS, COLS, seed, outliers=("channels", 0.005, 30.0))
    job = {"x": x,
           "codes": torch.empty((ROWS, COLS), dtype=torch.uint8, device="cuda"),
           "scales": torch.empty((ROWS, COLS // BLOCK), dtype=torch.float32, device="cuda"),
           "xhat": torch.empty((ROWS, COLS), dtype=torch.bfloat16, device="cuda"),
           "ssx": torch.empty(ROWS, dtype=torch.float32, device="cuda"),
           "sse": torch.empty(ROWS, dtype=torch.float32, device="cuda"),
           "wc": torch.empty((K, M), dtype=torch.uint8, device="cuda"),
           "ws": torch.empty((K, M // BLOCK), dtype=torch.float32, device="cuda"),
           "dy": wl.normal_bf16_device(K, N, seed + 1, 0.02),
           "dw": torch.empty((M, N), dtype=torch.float32, device="cuda")}
    job["unit"] = hl.unit_desc(x=x, codes=job["codes"], scales=job["scales"], xhat=job["xhat"],
                               row_ss_x=job["ssx"], row_ss_err=job["sse"])
    xw = wl.activation_device(K, M, seed + 2)  # the wgrad's X, encoded once
    hl.hilore_compress([hl.unit_desc(x=xw, codes=job["wc"], scales=job["ws"])], CODE, BLOCK)
    torch.cuda.synchronize()
    return job


def run_job(hl, job, stream):
    hl.hilore_compress([job["unit"]], CODE, BLOCK, stream=stream)
    hl.hilore_decompress([job["unit"]], CODE, BLOCK, stream=stream)
    hl.hilore_dequant_wgrad(job["wc"], job["ws"], CODE, BLOCK, job["dy"], job["dw"], K, M, N,
                            stream=stream)


NAMES = ("codes", "scales", "xhat", "ssx", "sse", "dw")


def outputs(job):
    return [host(job[k]) for k in NAMES]


def test_two_threads_two_streams(hl):
    jobs = [make_job(hl, 700 + 10 * i) for i in range(2)]
    ref = []
    for job in jobs:
        run_job(hl, job, None)
        torch.cuda.synchronize()
        ref.append(outputs(job))
    streams = [torch.cuda.Stream() for _ in jobs]
    errors = []

    def worker(i):
        try:
            for _ in range(8):
                run_job(hl, jobs[i], streams[i].cuda_stream)
            streams[i].synchronize()
        except Exception as e:  # surfaced below
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(jobs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    torch.cuda.synchronize()
    for i, job in enumerate(jobs):
        for got, want, name in zip(outputs(job), ref[i], NAMES):
            assert_bytes_equal(got, want, f"job {i} {name}")
