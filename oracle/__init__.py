"""Plain CPU oracle of the HiLoRe hot path (test infrastructure only).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` import this package.  The GPU product path never does: the oracle
and the HIP library share no code, header or table.

The arithmetic lives in ``oracle.c`` (plain single-threaded C, fp32 where the
GPU must match bit for bit, fp64 for every tolerance-checked "truth" value);
this module only marshals numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

INT8 = 0
E4M3FN = 1
E4M3FN_CAST = 2  # the paper's literal codec: a plain cast, no scales

GCC_FLAGS = ["-O2", "-std=c11", "-Wall", "-Wextra", "-ffp-contract=off", "-fno-fast-math",
             "-fPIC", "-shared"]


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc (plain C, no FMA contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", *GCC_FLAGS, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64 = ctypes.c_int64
        i32 = ctypes.c_int
        f32 = ctypes.c_float
        f64 = ctypes.c_double
        sig = {
            "orc_bf16_to_f32": (f32, [ctypes.c_uint16]),
            "orc_bf16_rne": (ctypes.c_uint16, [f32]),
            "orc_e4m3fn_rne": (ctypes.c_uint8, [f32]),
            "orc_e4m3fn_decode": (f64, [ctypes.c_uint8]),
            "orc_e4m3fn_cast": (ctypes.c_uint8, [f32]),
            "orc_e4m3fn_cast_to_bf16": (ctypes.c_uint16, [ctypes.c_uint8]),
            "orc_e4m3fn_cast_array": (None, [P, i64, P]),
            "orc_code_value": (f32, [i32, ctypes.c_uint8]),
            "orc_bf16_rne_array": (None, [P, i64, P]),
            "orc_e4m3fn_rne_array": (None, [P, i64, P]),
            "orc_grpo_advantages": (None, [P, i32, i32, f32, P]),
            "orc_grpo_coeffs": (None, [P, P, P, P, P, i32, i32, i32, f32, f32, f64, f64,
                                       P, P, P, P]),
            "orc_grpo_loss": (f64, [P, P, P, P, P, i32, i32, f64, f64, f64]),
            "orc_quantize": (None, [P, i64, i64, i64, i32, i32, P, P]),
            "orc_dequantize": (None, [P, P, i64, i64, i32, i32, P]),
            "orc_row_stats": (None, [P, i64, P, i64, i64, P, P]),
            "orc_unit_exposure_risk": (None, [P, P, i64, P, P, i64, f64, f64, P, P, P]),
            "orc_wgrad": (None, [P, P, i32, i32, P, i64, i64, i64, i64, i64, i64, i64, i32, P]),
            "orc_wgrad_entries": (None, [P, P, i32, i32, P, i64, i64, i64, P, P, i64, i32, P]),
            "orc_allocate": (i32, [i32, P, P, P, P, P, P, P, f64, f64, i32, i32, P, P, P]),
            "orc_allocate_brute": (i32, [i32, P, P, P, P, P, P, P, f64, f64, i32, i32, P, P, P]),
            "orc_grad_rel_err": (f64, [P, P, i64, f64]),
            "orc_calibrate": (None, [i32, i32, i32, P, P, P, P, P, P]),
            "orc_risk_score": (None, [i32, P, i32, P, P, P, P]),
            "orc_update_sparsity": (f64, [P, P, P, P, i32, i32, f64, P]),
            "orc_swiglu_bwd": (None, [P, P, P, i64, P, P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _ptr(a):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


# ---------------------------------------------------------------- formats --
def bf16_to_f32(h):
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_rne(v):
    v = _c(v, np.float32).ravel()
    out = np.empty(v.size, dtype=np.uint16)
    lib().orc_bf16_rne_array(_ptr(v), v.size, _ptr(out))
    return out


def e4m3fn_rne(v):
    v = _c(v, np.float32).ravel()
    out = np.empty(v.size, dtype=np.uint8)
    lib().orc_e4m3fn_rne_array(_ptr(v), v.size, _ptr(out))
    return out


def e4m3fn_cast(v):
    v = _c(v, np.float32).ravel()
    out = np.empty(v.size, dtype=np.uint8)
    lib().orc_e4m3fn_cast_array(_ptr(v), v.size, _ptr(out))
    return out


def e4m3fn_cast_to_bf16(c: int) -> int:
    return lib().orc_e4m3fn_cast_to_bf16(int(c))


def e4m3fn_decode(c: int) -> float:
    return lib().orc_e4m3fn_decode(int(c))


def code_value(code: int, c: int) -> float:
    return lib().orc_code_value(int(code), int(c))


# ------------------------------------------------------------------- GRPO --
def grpo_advantages(rewards, P, G, adv_eps=1e-6):
    r = _c(rewards, np.float32)
    adv = np.empty(P * G, dtype=np.float32)
    lib().orc_grpo_advantages(_ptr(r), P, G, adv_eps, _ptr(adv))
    return adv


def grpo_coeffs(rewards, logp_new, logp_old, logp_ref, mask, P, G, T, clip_eps=0.2,
                adv_eps=1e-6, beta=0.0, n_norm=0.0):
    """Returns (adv f32[R], ratio f64[R*T], flags u8[R*T], coeff f64[R*T])."""
    n = P * G * T
    r = _c(rewards, np.float32)
    ln, lo = _c(logp_new, np.float32), _c(logp_old, np.float32)
    lr = _c(logp_ref, np.float32)
    m = _c(mask, np.uint8)
    adv = np.empty(P * G, dtype=np.float32)
    ratio = np.empty(n, dtype=np.float64)
    flags = np.empty(n, dtype=np.uint8)
    coeff = np.empty(n, dtype=np.float64)
    lib().orc_grpo_coeffs(_ptr(r), _ptr(ln), _ptr(lo), _ptr(lr), _ptr(m), P, G, T, clip_eps,
                          adv_eps, float(beta), float(n_norm), _ptr(adv), _ptr(ratio),
                          _ptr(flags), _ptr(coeff))
    return adv, ratio, flags, coeff


def grpo_loss(adv, logp_new_f64, logp_old, logp_ref, mask, R, T, clip_eps=0.2, beta=0.0,
              n_norm=0.0):
    a = _c(adv, np.float32)
    ln = _c(logp_new_f64, np.float64)
    lo = _c(logp_old, np.float32)
    lr = _c(logp_ref, np.float32)
    m = _c(mask, np.uint8)
    return lib().orc_grpo_loss(_ptr(a), _ptr(ln), _ptr(lo), _ptr(lr), _ptr(m), R, T,
                               float(clip_eps), float(beta), float(n_norm))


# ------------------------------------------------------------------ codec --
def quantize(x_u16, code, block, cols=None):
    """x_u16: uint16 [rows, ld] bf16 bits (ld = row stride); quantises the first
    ``cols`` columns of every row (all of them by default).  With the literal
    cast code the scales are None."""
    x = _c(x_u16, np.uint16)
    rows, ld = x.shape
    cols = ld if cols is None else cols
    codes = np.empty((rows, cols), dtype=np.uint8)
    scales = None if code == E4M3FN_CAST else np.empty((rows, cols // block), dtype=np.float32)
    lib().orc_quantize(_ptr(x), rows, cols, ld, code, block, _ptr(codes), _ptr(scales))
    return codes, scales


def dequantize(codes, scales, code, block):
    c = _c(codes, np.uint8)
    s = _c(scales, np.float32)
    rows, cols = c.shape
    xh = np.empty((rows, cols), dtype=np.uint16)
    lib().orc_dequantize(_ptr(c), _ptr(s), rows, cols, code, block, _ptr(xh))
    return xh


def row_stats(x_u16, xhat_u16):
    x = _c(x_u16, np.uint16)
    xh = _c(xhat_u16, np.uint16)
    rows, cols = xh.shape
    ss_x = np.empty(rows, dtype=np.float64)
    ss_e = np.empty(rows, dtype=np.float64)
    lib().orc_row_stats(_ptr(x), x.shape[1], _ptr(xh), rows, cols, _ptr(ss_x), _ptr(ss_e))
    return ss_x, ss_e


def unit_exposure_risk(coeff, mask, ss_x, ss_err, d_u, eps_alpha=1e-8, eps_rel=1e-8):
    w = _c(coeff, np.float64)
    m = _c(mask, np.uint8)
    sx = _c(ss_x, np.float64)
    se = _c(ss_err, np.float64)
    e = ctypes.c_double()
    k = ctypes.c_double()
    rel = ctypes.c_double()
    lib().orc_unit_exposure_risk(_ptr(w), _ptr(m), sx.size, _ptr(sx), _ptr(se), int(d_u),
                                 float(eps_alpha), float(eps_rel), ctypes.byref(e),
                                 ctypes.byref(k), ctypes.byref(rel))
    return e.value, k.value, rel.value


# ------------------------------------------------------------------ wgrad --
def wgrad(codes, scales, code, block, dy_u16, i0=0, i1=None, j0=0, j1=None, variant=0):
    c = _c(codes, np.uint8)
    s = _c(scales, np.float32)
    d = _c(dy_u16, np.uint16)
    K, M = c.shape
    N = d.shape[1]
    i1 = M if i1 is None else i1
    j1 = N if j1 is None else j1
    out = np.empty((i1 - i0, j1 - j0), dtype=np.float64)
    lib().orc_wgrad(_ptr(c), _ptr(s), code, block, _ptr(d), K, M, N, i0, i1, j0, j1, variant,
                    _ptr(out))
    return out


def wgrad_entries(codes, scales, code, block, dy_u16, ii, jj, variant=0, K=None):
    c = _c(codes, np.uint8)
    s = _c(scales, np.float32)
    d = _c(dy_u16, np.uint16)
    Kc, M = c.shape
    N = d.shape[1]
    ii = _c(ii, np.int64)
    jj = _c(jj, np.int64)
    out = np.empty(ii.size, dtype=np.float64)
    lib().orc_wgrad_entries(_ptr(c), _ptr(s), code, block, _ptr(d), Kc if K is None else K, M,
                            N, _ptr(ii), _ptr(jj), ii.size, variant, _ptr(out))
    return out


# ------------------------------------------------------------- allocation --
ACT_R, ACT_H, ACT_L = 0, 1, 2


def allocate(q, verified, tau_h, tau_l, dm_h, dm_l, psi, m_res, delta_b, n_b=1024, n_d=1024,
             brute=False):
    """Joint H/L/R allocation of App. B.2 (dynamic programme, or brute force
    over 3^U with brute=True).  Returns (action u8[U], totals f64[3] =
    (utility, memory, risk), jk i64[2] = terminal integer costs)."""
    q = _c(q, np.uint8)
    v = _c(verified, np.uint8)
    arrs = [_c(a, np.float64) for a in (tau_h, tau_l, dm_h, dm_l, psi)]
    U = q.size
    action = np.zeros(max(U, 1), dtype=np.uint8)
    totals = np.zeros(3, dtype=np.float64)
    jk = np.zeros(2, dtype=np.int64)
    fn = lib().orc_allocate_brute if brute else lib().orc_allocate
    rc = fn(U, _ptr(q), _ptr(v), *[_ptr(a) for a in arrs], float(m_res), float(delta_b),
            int(n_b), int(n_d), _ptr(action), _ptr(totals), _ptr(jk))
    if rc != 0:
        raise ValueError("invalid allocation arguments")
    return action[:U], totals, jk


# ------------------------------------------------- calibration and diagnostics --
def grad_rel_err(g_l, g_ex, eps_num=1e-30):
    """y = sqrt(||g_l - g_ex||^2 / max(||g_ex||^2, eps_num)) over fp32 values, fp64 sums."""
    a = _c(g_l, np.float32).ravel()
    b = _c(g_ex, np.float32).ravel()
    assert a.size == b.size
    return lib().orc_grad_rel_err(_ptr(a), _ptr(b), a.size, float(eps_num))


def calibrate(unit_class, exposure, rel_err, grad_err, n_classes):
    """exposure, rel_err, grad_err: [n_batches, n_units] (fp32 values).
    Returns (kappa f64[n_classes], ebar f64[n_units])."""
    cls = _c(unit_class, np.int32).ravel()
    e = _c(exposure, np.float32)
    r = _c(rel_err, np.float32)
    y = _c(grad_err, np.float32)
    nb, nu = e.shape
    assert cls.size == nu and r.shape == e.shape and y.shape == e.shape
    kappa = np.empty(max(n_classes, 1), dtype=np.float64)
    ebar = np.empty(max(nu, 1), dtype=np.float64)
    lib().orc_calibrate(nu, nb, int(n_classes), _ptr(cls), _ptr(e), _ptr(r), _ptr(y),
                        _ptr(kappa), _ptr(ebar))
    return kappa[:n_classes], ebar[:nu]


def risk_score(unit_class, kappa, ebar, exposure):
    cls = _c(unit_class, np.int32).ravel()
    k = _c(kappa, np.float64).ravel()
    eb = _c(ebar, np.float64).ravel()
    e = _c(exposure, np.float32).ravel()
    psi = np.empty(max(cls.size, 1), dtype=np.float64)
    lib().orc_risk_score(cls.size, _ptr(cls), k.size, _ptr(k), _ptr(eb), _ptr(e), _ptr(psi))
    return psi[:cls.size]


def update_sparsity(coeff, flags, adv, mask, R, T, top_frac=0.1):
    """Returns (counts i64[3] = padding, zero-advantage, clipped slots; top-k share)."""
    w = _c(coeff, np.float64).ravel()
    f = _c(flags, np.uint8).ravel()
    a = _c(adv, np.float32).ravel()
    m = _c(mask, np.uint8)
    counts = np.zeros(3, dtype=np.int64)
    share = lib().orc_update_sparsity(_ptr(w), _ptr(f), _ptr(a), None if m is None else _ptr(m.ravel()),
                                      int(R), int(T), float(top_frac), _ptr(counts))
    return counts, share


def lora_down_grad(codes, scales, code, block, dh_u16, scale=1.0, variant=0):
    """Gradient of the LoRA down-projection weight A [r, in] of a linear layer
    whose saved input X [K, in] is an L unit: with h = X A^T, z = h B^T and
    the layer output y = X W^T + scale * z (PEFT's convention, scale = alpha/r),
    dA = scale * (G B)^T X = scale * dh^T X with dh = G B [K, r].  This is the
    weight gradient X^T dh of orc_wgrad, transposed and scaled."""
    return scale * wgrad(codes, scales, code, block, dh_u16, variant=variant).T


def swiglu_bwd(g, u, dh):
    """Backward of h = silu(g) * u in fp64: returns (dg, du) with the shape of g."""
    g64 = _c(g, np.float64)
    u64 = _c(u, np.float64)
    d64 = _c(dh, np.float64)
    assert g64.shape == u64.shape == d64.shape
    dg = np.empty(g64.shape, dtype=np.float64)
    du = np.empty(g64.shape, dtype=np.float64)
    lib().orc_swiglu_bwd(_ptr(g64), _ptr(u64), _ptr(d64), g64.size, _ptr(dg), _ptr(du))
    return dg, du
