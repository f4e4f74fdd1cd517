"""Seeded synthetic inputs for the HiLoRe hot path.

This module only draws random numbers.  It holds none of the method's
arithmetic (no advantages, ratios, coefficients, quantisation or reductions),
so both the GPU path and the CPU oracle can take their inputs from it.

The paper trains on rollouts of real models (DeepMath10K, TACO-Verified,
Knights-and-Knaves); none of those datasets or weights are used.  The
synthetic inputs below stand in for them with the shapes, sizes and value
distributions of the workloads: binary rewards, groups of G responses,
per-token log-probabilities near -2 with a small policy drift, bf16
activations of decoder layers with heavy channels, and a length mask for
padded responses (App. D.1.1 and Table execution-configurations).

Host generators use numpy's PCG64 and return numpy arrays (bf16 values as
uint16 bit patterns); device generators use torch's generator on the GPU and
return torch tensors, for the full-size workloads that would take too long to
draw on the host.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence, Tuple

import numpy as np

BASE_SEED = 2026  # the paper's split and pilot seed (App. D.1.1)


def rng(seed: int, *stream: int) -> np.random.Generator:
    """PCG64 generator for (seed, stream...)."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=stream)))


def to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """Round an fp32 array to bf16 (torch's cast) and return the uint16 bits."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


# --------------------------------------------------------------------- GRPO --
@dataclasses.dataclass
class GrpoBatch:
    P: int
    G: int
    T: int
    rewards: np.ndarray            # f32 [P*G], values in {0, 1}
    logp_new: np.ndarray           # f32 [P*G*T]
    logp_old: np.ndarray           # f32 [P*G*T]
    logp_ref: Optional[np.ndarray]  # f32 [P*G*T] or None
    mask: Optional[np.ndarray]     # u8 [P*G*T] or None (all valid)


def pad_lengths(R: int, T: int, frac: float, g: np.random.Generator) -> np.ndarray:
    """Per-response trailing-padding lengths: pad_j = floor(0.6 T u_j) with
    u_j ~ U(0,1), then adjusted from the last response backwards so that the
    total equals round(frac R T)."""
    pad = np.floor(0.6 * T * g.random(R)).astype(np.int64)
    diff = int(round(frac * R * T)) - int(pad.sum())
    j = R - 1
    while diff != 0:
        step = min(diff, T - int(pad[j])) if diff > 0 else -min(-diff, int(pad[j]))
        pad[j] += step
        diff -= step
        j = (j - 1) % R
    return pad


def grpo_batch(P: int, G: int, T: int, seed: int, delta_sigma: float = 0.05,
               with_ref: bool = False, pad_frac: Optional[float] = None,
               reward_p: float = 0.5) -> GrpoBatch:
    """Binary rewards ~ Bernoulli(reward_p); s_old ~ N(-2, 0.5);
    s_new = s_old + N(0, delta_sigma); optional s_ref = s_old + N(0, 0.05);
    optional length mask with a fraction pad_frac of slots padded."""
    R = P * G
    g = rng(seed, 1)
    rewards = (g.random(R) < reward_p).astype(np.float32)
    old = g.normal(-2.0, 0.5, R * T).astype(np.float32)
    new = (old.astype(np.float64) + g.normal(0.0, delta_sigma, R * T)).astype(np.float32)
    ref = None
    if with_ref:
        ref = (old.astype(np.float64) + g.normal(0.0, 0.05, R * T)).astype(np.float32)
    mask = None
    if pad_frac is not None:
        pad = pad_lengths(R, T, pad_frac, g)
        t = np.arange(T)[None, :]
        mask = (t < (T - pad)[:, None]).astype(np.uint8).ravel()
    return GrpoBatch(P, G, T, rewards, new, old, ref, mask)


def grpo_batch_device(P: int, G: int, T: int, seed: int, delta_sigma: float = 0.05,
                      pad_frac: Optional[float] = None, device="cuda"):
    """Device-side GRPO inputs with grpo_batch's recipe (Bernoulli(0.5) rewards,
    s_old ~ N(-2, 0.5), s_new = s_old + N(0, delta_sigma), trailing padding of
    a fraction pad_frac drawn by pad_lengths), drawn with torch's generator in
    fp32 for batches too large to draw on the host.  Returns (rewards,
    logp_new, logp_old, mask or None) as device tensors; the values differ from
    grpo_batch's for the same seed."""
    import torch

    R = P * G
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    rewards = (torch.rand(R, generator=gen, device=device) < 0.5).to(torch.float32)
    old = torch.randn(R * T, generator=gen, device=device).mul_(0.5).sub_(2.0)
    new = torch.randn(R * T, generator=gen, device=device).mul_(delta_sigma).add_(old)
    mask = None
    if pad_frac is not None:
        pad = torch.from_numpy(pad_lengths(R, T, pad_frac, rng(seed, 1))).to(device)
        t = torch.arange(T, device=device)
        mask = (t[None, :] < (T - pad)[:, None]).to(torch.uint8).reshape(-1)
    return rewards, new, old, mask


# -------------------------------------------------------------- activations --
def activation_host(rows: int, cols: int, seed: int, dist: str = "normal",
                    outliers: Optional[Tuple[str, float, float]] = None,
                    ld: Optional[int] = None) -> np.ndarray:
    """bf16 activation [rows, ld] (uint16 bits; columns >= cols are filled with
    unrelated values when ld > cols).

    dist: "normal" (N(0,1)) or "student_t3" (Student-t, nu = 3).
    outliers: ("entries", frac, factor): round(frac * rows * cols) distinct
              entries chosen uniformly are multiplied by factor;
              ("channels", frac, factor): round(frac * cols) distinct whole
              columns are multiplied by factor."""
    g = rng(seed, 2)
    ld = cols if ld is None else ld
    if dist == "normal":
        x = g.standard_normal((rows, ld), dtype=np.float32)
    elif dist == "student_t3":
        x = g.standard_t(3, (rows, ld)).astype(np.float32)
    else:
        raise ValueError(dist)
    if outliers is not None:
        kind, frac, factor = outliers
        if kind == "entries":
            k = int(round(frac * rows * cols))
            idx = g.choice(rows * cols, size=k, replace=False)
            r, c = np.divmod(idx, cols)
            x[r, c] *= np.float32(factor)
        elif kind == "channels":
            ch = channel_outliers(cols, frac, seed)
            x[:, ch] *= np.float32(factor)
        else:
            raise ValueError(kind)
    return to_bf16_bits(x)


def channel_outliers(cols: int, frac: float, seed: int) -> np.ndarray:
    """round(frac * cols) distinct column indices (seeded)."""
    g = rng(seed, 3)
    return np.sort(g.choice(cols, size=int(round(frac * cols)), replace=False))


def normal_bf16_host(rows: int, cols: int, seed: int, sigma: float) -> np.ndarray:
    g = rng(seed, 4)
    return to_bf16_bits((g.standard_normal((rows, cols)) * sigma).astype(np.float32))


def activation_device(rows: int, cols: int, seed: int, dist: str = "normal",
                      outliers: Optional[Tuple[str, float, float]] = None,
                      device="cuda", chunk_rows: int = 8192, out=None):
    """Device-side bf16 activation [rows, cols] drawn with torch's generator
    (for sizes too large to draw on the host).  Same recipes as
    activation_host except that entry outliers are not offered; the values
    differ from activation_host's for the same seed."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    x = out if out is not None else torch.empty((rows, cols), dtype=torch.bfloat16,
                                                   device=device)
    ch = None
    factor = 1.0
    if outliers is not None:
        kind, frac, factor = outliers
        if kind != "channels":
            raise ValueError("device generator offers channel outliers only")
        ch = torch.from_numpy(channel_outliers(cols, frac, seed)).to(device)
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        z = torch.randn((r1 - r0, cols), generator=gen, device=device, dtype=torch.float32)
        if dist == "student_t3":
            n = torch.randn((3, r1 - r0, cols), generator=gen, device=device,
                            dtype=torch.float32)
            z.mul_(torch.rsqrt(n.square().sum(0).div_(3.0)))
            del n
        elif dist != "normal":
            raise ValueError(dist)
        if ch is not None:
            z[:, ch] *= factor
        x[r0:r1].copy_(z)
        del z
    return x


def normal_bf16_device(rows: int, cols: int, seed: int, sigma: float, device="cuda"):
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    return (torch.randn((rows, cols), generator=gen, device=device, dtype=torch.float32)
            .mul_(sigma).to(torch.bfloat16))


# ------------------------------------------------------------ workload table --
@dataclasses.dataclass(frozen=True)
class UnitShape:
    name: str
    rows: int
    cols: int


@dataclasses.dataclass(frozen=True)
class Workload:
    """One of the five synthetic workloads (sizes as named)."""
    key: str
    description: str
    P: int
    G: int
    T: int
    units: Tuple[UnitShape, ...]
    code: str             # "int8" | "e4m3fn"
    block: int
    dist: str
    outliers: Optional[Tuple[str, float, float]]
    pad_frac: Optional[float] = None
    wgrad: Optional[Tuple[int, int, int]] = None   # (K, M, N)

    @property
    def seed(self) -> int:
        return BASE_SEED + {"tiny": 1, "qwen2_7b_layer": 2, "qwen2_7b_plan": 3,
                            "wgrad_4096": 4, "llama3_8b_stress": 5}[self.key]


TINY = Workload(
    "tiny", "GRPO 4 prompts x 8 responses x 32 tokens; one 1024x896 bf16 activation "
    "(N(0,1), 1% of entries x20), int8 1x128", 4, 8, 32,
    (UnitShape("act", 1024, 896),), "int8", 128, "normal", ("entries", 0.01, 20.0))

QWEN2_7B_LAYER = Workload(
    "qwen2_7b_layer", "Qwen2-7B-width layer, 8 responses x 2048 tokens: hidden 16384x3584 "
    "and MLP intermediate 16384x18944 bf16 (N(0,1), 0.5% channels x30), fp8-e4m3 1x128",
    1, 8, 2048, (UnitShape("hidden", 16384, 3584), UnitShape("mlp", 16384, 18944)),
    "e4m3fn", 128, "normal", ("channels", 0.005, 30.0))

QWEN2_7B_PLAN = Workload(
    "qwen2_7b_plan", "whole-model plan, 28 layers x 7 units of 16384x3584 bf16; seeded "
    "40% L (int8 1x64) / 30% H / 30% R", 1, 8, 2048,
    tuple(UnitShape(f"l{l}u{u}", 16384, 3584) for l in range(28) for u in range(7)),
    "int8", 64, "normal", ("channels", 0.005, 30.0))

WGRAD_4096 = Workload(
    "wgrad_4096", "fused dequant weight gradient: X fp8-e4m3 1x128 16384x4096, dY bf16 "
    "16384x4096 N(0,0.02^2), dW fp32 4096x4096", 1, 8, 2048,
    (UnitShape("x", 16384, 4096),), "e4m3fn", 128, "normal", None,
    wgrad=(16384, 4096, 4096))

LLAMA3_8B_STRESS = Workload(
    "llama3_8b_stress", "Llama-3-8B-shaped stress: 32 MLP intermediates 32768x14336 bf16 "
    "(Student-t nu=3), int8 1x128; GRPO 2 prompts x 16 responses, 30% padded", 2, 16, 1024,
    tuple(UnitShape(f"l{l}mlp", 32768, 14336) for l in range(32)), "int8", 128,
    "student_t3", None, pad_frac=0.3)

WORKLOADS = {w.key: w for w in (TINY, QWEN2_7B_LAYER, QWEN2_7B_PLAN, WGRAD_4096,
                                LLAMA3_8B_STRESS)}


def plan_actions(n_units: int, seed: int, frac_l: float = 0.4, frac_h: float = 0.3) -> np.ndarray:
    """Seeded H/L/R assignment: a permutation puts round(frac_l * n) units in L,
    round(frac_h * n) in H and the rest in R.  Returns an array of 'H'/'L'/'R'."""
    g = rng(seed, 5)
    perm = g.permutation(n_units)
    n_l = int(round(frac_l * n_units))
    n_h = int(round(frac_h * n_units))
    act = np.full(n_units, "R", dtype="<U1")
    act[perm[:n_l]] = "L"
    act[perm[n_l:n_l + n_h]] = "H"
    return act


# ------------------------------------------------------ allocation instances --
@dataclasses.dataclass
class AllocInstance:
    """Inputs of one H/L/R allocation (App. B.2): per unit the retained
    representation q (0 = R, 1 = H, 2 = L), the verified-action bit mask
    (bit a for action a), the utilities and memory costs of H and L, and the
    risk psi of L; the memory and risk budgets of the microbatch."""
    q: np.ndarray
    verified: np.ndarray
    tau_h: np.ndarray
    tau_l: np.ndarray
    dm_h: np.ndarray
    dm_l: np.ndarray
    psi: np.ndarray
    m_res: float
    delta_b: float

    @property
    def U(self) -> int:
        return int(self.q.size)

    def arrays(self):
        return (self.q, self.verified, self.tau_h, self.tau_l, self.dm_h, self.dm_l, self.psi)


def alloc_instance(shapes: Sequence[Tuple[int, int]], seed: int, block: int = 128,
                   frac_q: Tuple[float, float, float] = (0.15, 0.6, 0.25),
                   mem_frac: float = 0.3, risk_frac: float = 0.25) -> AllocInstance:
    """Synthetic profiled units of the given (rows, cols) bf16 shapes.  H keeps
    the tensor (2 B per element), L its codes and scales (1 + 4/block B); the
    H utility is the recompute time saved, drawn around the time to stream the
    tensor at 1.5 TB/s (x U(0.6, 1.6)); L saves the same minus a codec cost of
    3 B per element at 5 TB/s (x U(0.8, 1.2)), so a few L utilities are not
    positive; psi ~ lognormal(-7, 1.5).  q is R/H/L with probabilities frac_q;
    10% of the units lack a verified L.  Budgets: mem_frac of the total H
    memory and risk_frac of the total psi."""
    g = rng(seed, 6)
    U = len(shapes)
    n = np.array([r * c for r, c in shapes], dtype=np.float64)
    dm_h = 2.0 * n
    dm_l = n * (1.0 + 4.0 / block)
    tau_h = dm_h / 1.5e12 * g.uniform(0.6, 1.6, U)
    tau_l = tau_h - 3.0 * n / 5e12 * g.uniform(0.8, 1.2, U)
    psi = g.lognormal(-7.0, 1.5, U)
    q = g.choice(3, size=U, p=np.asarray(frac_q) / np.sum(frac_q)).astype(np.uint8)
    verified = np.where(g.random(U) < 0.1, 0b011, 0b111).astype(np.uint8)
    return AllocInstance(q, verified, tau_h, tau_l, dm_h, dm_l, psi,
                         float(mem_frac * dm_h.sum()), float(risk_frac * psi.sum()))


def alloc_small(U: int, seed: int, integer: bool = False, scale: float = 16.0) -> AllocInstance:
    """Small random instance for exhaustive checks: memory costs and psi of a
    few grid steps (so that budgets bind), utilities real or small integers
    (integers make many exact ties)."""
    g = rng(seed, 7)
    if integer:
        tau_h = g.integers(1, 4, U).astype(np.float64)
        tau_l = g.integers(0, 4, U).astype(np.float64)
    else:
        tau_h = g.uniform(0.1, 2.0, U)
        tau_l = g.uniform(-0.2, 2.0, U)
    dm_h = g.uniform(0.0, scale, U) * (g.random(U) < 0.9)
    dm_l = dm_h * g.uniform(0.3, 0.7, U)
    psi = g.uniform(0.0, scale, U) * (g.random(U) < 0.9)
    q = g.choice(3, size=U, p=[0.2, 0.55, 0.25]).astype(np.uint8)
    verified = np.where(g.random(U) < 0.15, 0b011, 0b111).astype(np.uint8)
    return AllocInstance(q, verified, tau_h, tau_l, dm_h, dm_l, psi,
                         float(g.uniform(0.2, 0.6) * dm_h.sum()),
                         float(g.uniform(0.2, 0.6) * psi.sum()))


def qwen2_7b_unit_mix(layers: int = 28, tokens: int = 16384) -> Tuple[Tuple[int, int], ...]:
    """Per decoder layer 4 hidden-width (3584) and 3 MLP-width (18944) saved
    activations of the microbatch: 196 units for 28 layers."""
    return tuple((tokens, c) for _ in range(layers) for c in (3584,) * 4 + (18944,) * 3)
