"""Helpers shared by the GPU parity tests: host <-> device copies and the
tolerance rule.

Tolerance for floating-point outputs: |gpu - truth| <= 1e-5 * |truth|
(truth in fp64 from the oracle) where nothing cancels: ratios, and update
coefficients without the KL term (each a single product of rounded factors).
Where terms of opposite sign can cancel (coefficients with the K3 KL term,
whose policy and KL parts may nearly annul) or an fp32 sum is compared with
its fp64 value (row sums, exposure, risk, relative error), the absolute error
is bounded instead by 1e-5 * max(|truth|, 1e-3 * max|truth|): an element far
below the largest carries the rounding of the terms it was formed from, not
its own.  Bit-exact outputs (advantages, flags, codes, scales,
reconstructions) are compared as raw bytes.
"""
import numpy as np
import torch

REL_TOL = 1e-5


def dev(a: np.ndarray) -> torch.Tensor:
    """numpy -> torch CUDA tensor with the same bytes (uint16 -> bfloat16)."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def host(t: torch.Tensor) -> np.ndarray:
    """torch tensor -> numpy with the same bytes (bfloat16 -> uint16)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float8_e4m3fn:
        return t.view(torch.uint8).numpy()
    return t.numpy()


def empty(shape, dtype) -> torch.Tensor:
    if isinstance(shape, int):
        shape = (shape,)
    return torch.empty(shape, dtype=dtype, device="cuda")


def filled(shape, dtype, value=0) -> torch.Tensor:
    """A buffer pre-filled with a sentinel so unwritten outputs are noticed."""
    if isinstance(shape, int):
        shape = (shape,)
    return torch.full(shape, value, dtype=dtype, device="cuda")


def assert_close(gpu, truth, what="", rel=REL_TOL, floor_frac=1e-3):
    """floor_frac = 0: a pure relative check (see the module docstring)."""
    gpu = np.asarray(gpu, dtype=np.float64)
    truth = np.asarray(truth, dtype=np.float64)
    assert gpu.shape == truth.shape, what
    if truth.size == 0:
        return
    floor = floor_frac * np.abs(truth).max()
    err = np.abs(gpu - truth)
    lim = rel * np.maximum(np.abs(truth), floor)
    bad = err > lim
    if bad.any():
        i = int(np.argmax(err / np.maximum(lim, 1e-300)))
        raise AssertionError(f"{what}: {bad.sum()} of {truth.size} outside tolerance; worst at "
                             f"{i}: gpu={gpu.flat[i]!r} truth={truth.flat[i]!r}")


def assert_bytes_equal(gpu, ref, what=""):
    gpu = np.ascontiguousarray(gpu)
    ref = np.ascontiguousarray(ref)
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    g8 = gpu.view(np.uint8)
    r8 = ref.view(np.uint8)
    if not np.array_equal(g8, r8):
        diff = np.nonzero(gpu.reshape(-1).view(np.uint8 if gpu.dtype.itemsize == 1 else
                                               {2: np.uint16, 4: np.uint32}[gpu.dtype.itemsize])
                          != ref.reshape(-1).view(np.uint8 if ref.dtype.itemsize == 1 else
                                                  {2: np.uint16, 4: np.uint32}[ref.dtype.itemsize]))[0]
        i = int(diff[0])
        raise AssertionError(f"{what}: {diff.size} elements differ; first at flat index {i}: "
                             f"gpu={gpu.reshape(-1)[i]!r} ref={ref.reshape(-1)[i]!r}")


def rel_fro(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))
