"""Thin Python binding of libhilore (the C-ABI in include/hilore.h).

Argument marshalling only: every step runs in the library's HIP kernels.
Tensors are torch tensors on the GPU (torch provides device memory and the
stream); each function passes their data pointers and the current stream to
the C entry point of the same name and raises HiloreError on a non-zero
status.  There is no fallback: without libhilore.so the import fails.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

from . import defaults as _d

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhilore.so")

HILORE_OK = 0
HILORE_ERR_INVALID_ARG = 1
HILORE_ERR_ALIGNMENT = 2
HILORE_ERR_UNSUPPORTED = 3
HILORE_ERR_WORKSPACE = 4
HILORE_ERR_HIP = 5

HILORE_CODE_INT8 = 0
HILORE_CODE_FP8_E4M3FN = 1
HILORE_CODE_FP8_E4M3FN_CAST = 2  # the paper's literal codec: plain cast, no scales, block 0
CODES = {"int8": HILORE_CODE_INT8, "e4m3fn": HILORE_CODE_FP8_E4M3FN,
         "e4m3fn_cast": HILORE_CODE_FP8_E4M3FN_CAST}


class HiloreError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {status_string(status)} ({status})")


class hilore_unit_desc(ctypes.Structure):
    _fields_ = [
        ("x", ctypes.c_void_p),
        ("codes", ctypes.c_void_p),
        ("scales", ctypes.c_void_p),
        ("xhat", ctypes.c_void_p),
        ("row_ss_x", ctypes.c_void_p),
        ("row_ss_err", ctypes.c_void_p),
        ("rows", ctypes.c_int64),
        ("cols", ctypes.c_int64),
        ("ld", ctypes.c_int64),
    ]


_lib = None


def load() -> ctypes.CDLL:
    """Load libhilore.so (built in-tree by __graft_entry__.build())."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i32 = ctypes.c_int
    i64 = ctypes.c_int64
    f32 = ctypes.c_float
    f64 = ctypes.c_double
    sig = {
        "hilore_status_string": (ctypes.c_char_p, [i32]),
        "hilore_version": (i32, []),
        "hilore_grpo_coeffs_workspace_bytes": (ctypes.c_size_t, [i32, i32, i32]),
        "hilore_grpo_coeffs": (i32, [P, P, P, P, P, i32, i32, i32, f32, f32, f32, f64,
                                     P, P, P, P, P, ctypes.c_size_t, P]),
        "hilore_compress": (i32, [P, i32, i32, i32, P]),
        "hilore_decompress": (i32, [P, i32, i32, i32, P]),
        "hilore_unit_exposure_risk_workspace_bytes": (ctypes.c_size_t, [i64, i32]),
        "hilore_unit_exposure_risk": (i32, [P, P, i64, P, i32, f32, f32, P, P, P, P,
                                            ctypes.c_size_t, P]),
        "hilore_unit_exposure_risk_noalloc": (i32, [P, P, i64, P, i32, f32, f32, P, P, P, P]),
        "hilore_dequant_wgrad": (i32, [P, P, i32, i32, P, P, i64, i64, i64, i32, P]),
        "hilore_allocate_workspace_bytes": (ctypes.c_size_t, [i32, i32, i32]),
        "hilore_allocate": (i32, [i32, P, P, P, P, P, P, P, f64, f64, i32, i32, P, P, P, P,
                                  ctypes.c_size_t, P]),
        "hilore_lora_grad_workspace_bytes": (ctypes.c_size_t, [i64, i64, i32]),
        "hilore_dequant_lora_grad": (i32, [P, P, i32, i32, P, P, i64, i64, i32, f32, i32, P,
                                           ctypes.c_size_t, P]),
        "hilore_dequant_swiglu_bwd": (i32, [P, P, i32, i32, P, P, P, P]),
        "hilore_grad_rel_err_workspace_bytes": (ctypes.c_size_t, [i64]),
        "hilore_grad_rel_err": (i32, [P, P, i64, f64, P, P, ctypes.c_size_t, P]),
        "hilore_calibrate": (i32, [i32, i32, i32, P, P, P, P, P, P, P]),
        "hilore_risk_score": (i32, [i32, P, i32, P, P, P, P, P]),
        "hilore_update_sparsity": (i32, [P, P, P, P, i32, i32, f64, P, P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def status_string(status: int) -> str:
    return load().hilore_status_string(int(status)).decode()


def version() -> int:
    return load().hilore_version()


def _check(fn: str, status: int) -> None:
    if status != HILORE_OK:
        raise HiloreError(fn, status)


def _device(t) -> None:
    if not t.is_cuda:
        raise ValueError(f"libhilore takes device tensors, got one on {t.device}")


def _p(t) -> Optional[int]:
    """Data pointer of a dense device tensor (None -> NULL).  A host tensor
    would hand the kernels a host address and a strided view the wrong
    elements, so both are refused here."""
    if t is None:
        return None
    _device(t)
    if not t.is_contiguous():
        raise ValueError(f"libhilore takes dense tensors, got strides {tuple(t.stride())}")
    return t.data_ptr()


def _p_rows(t) -> Optional[int]:
    """Data pointer of a row-strided 2-D device tensor (a unit's bf16 x: rows
    may be padded, elements within a row are contiguous)."""
    if t is None:
        return None
    _device(t)
    if t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError(f"x must be 2-D with contiguous rows, got strides {tuple(t.stride())}")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return int(stream)
    import torch

    return torch.cuda.current_stream().cuda_stream


def _code(code) -> int:
    return CODES[code] if isinstance(code, str) else int(code)


def unit_desc(x=None, codes=None, scales=None, xhat=None, row_ss_x=None, row_ss_err=None,
              rows=None, cols=None, ld=None) -> hilore_unit_desc:
    """Descriptor of one unit from torch tensors (shapes taken from the tensors
    when not given: x is [rows, ld] with ld = row stride; codes [rows, cols])."""
    ref = x if x is not None else (codes if codes is not None else xhat)
    if rows is None:
        rows = ref.shape[0] if ref is not None else (row_ss_x.shape[0] if row_ss_x is not None else 0)
    if cols is None:
        if codes is not None:
            cols = codes.shape[1]
        elif xhat is not None:
            cols = xhat.shape[1]
        else:
            cols = x.shape[1]
    if ld is None:
        ld = x.stride(0) if x is not None else cols
    return hilore_unit_desc(_p_rows(x), _p(codes), _p(scales), _p(xhat), _p(row_ss_x),
                            _p(row_ss_err), int(rows), int(cols), int(ld))


def _desc_array(units: Sequence[hilore_unit_desc]):
    arr = (hilore_unit_desc * max(1, len(units)))(*units)
    return arr, len(units)


# ---------------------------------------------------------------- entry points --
def _workspace(workspace, nbytes: int, stream):
    """(pointer, size) of a caller's workspace tensor; without one, a fresh
    zeroed device buffer of the queried size (torch's allocator) when any is
    needed.  torch reuses a freed buffer in the order of its current stream, so
    a call on another stream must bring its own workspace."""
    if workspace is None:
        if nbytes == 0:
            return None, 0, None
        if stream is not None:
            raise ValueError("a call on an explicit stream needs an explicit workspace")
        import torch

        workspace = torch.zeros(nbytes, dtype=torch.uint8, device="cuda")
    return _p(workspace), workspace.numel() * workspace.element_size(), workspace


def hilore_grpo_coeffs_workspace_bytes(P: int, G: int, T: int) -> int:
    return int(load().hilore_grpo_coeffs_workspace_bytes(int(P), int(G), int(T)))


def hilore_grpo_coeffs(rewards, logp_new, logp_old, logp_ref, mask, P, G, T, clip_eps,
                       adv_eps, beta, n_norm, adv, ratio, flags, coeff, workspace=None,
                       stream=None):
    """workspace: a device tensor of at least hilore_grpo_coeffs_workspace_bytes(P, G, T)
    bytes, or None (a buffer of that size is then taken from torch's allocator when
    the call counts N)."""
    need = (hilore_grpo_coeffs_workspace_bytes(P, G, T)
            if mask is not None and float(n_norm) <= 0.0 else 0)
    wp, wb, _keep = _workspace(workspace, need, stream)
    st = load().hilore_grpo_coeffs(_p(rewards), _p(logp_new), _p(logp_old), _p(logp_ref),
                                   _p(mask), int(P), int(G), int(T), float(clip_eps),
                                   float(adv_eps), float(beta), float(n_norm), _p(adv),
                                   _p(ratio), _p(flags), _p(coeff), wp, wb, _stream(stream))
    _check("hilore_grpo_coeffs", st)


def hilore_compress(units: Sequence[hilore_unit_desc], code, block: int, stream=None):
    arr, n = _desc_array(units)
    _check("hilore_compress",
           load().hilore_compress(arr, n, _code(code), int(block), _stream(stream)))


def hilore_decompress(units: Sequence[hilore_unit_desc], code, block: int, stream=None):
    arr, n = _desc_array(units)
    _check("hilore_decompress",
           load().hilore_decompress(arr, n, _code(code), int(block), _stream(stream)))


def hilore_unit_exposure_risk_workspace_bytes(rows: int, n_units: int) -> int:
    return int(load().hilore_unit_exposure_risk_workspace_bytes(int(rows), int(n_units)))


def hilore_unit_exposure_risk(coeff, mask, rows: int, units: Sequence[hilore_unit_desc],
                              eps_alpha: float, eps_rel: float, exposure, risk, rel_err,
                              workspace=None, stream=None):
    """workspace: a device tensor of at least
    hilore_unit_exposure_risk_workspace_bytes(rows, len(units)) bytes, or None (a
    buffer of that size is then taken from torch's allocator)."""
    arr, n = _desc_array(units)
    wp, wb, _keep = _workspace(workspace, hilore_unit_exposure_risk_workspace_bytes(rows, n),
                               stream)
    _check("hilore_unit_exposure_risk",
           load().hilore_unit_exposure_risk(_p(coeff), _p(mask), int(rows), arr, n,
                                            float(eps_alpha), float(eps_rel), _p(exposure),
                                            _p(risk), _p(rel_err), wp, wb, _stream(stream)))


def hilore_unit_exposure_risk_noalloc(coeff, mask, rows: int, units: Sequence[hilore_unit_desc],
                                      eps_alpha: float, eps_rel: float, exposure, risk, rel_err,
                                      stream=None):
    """hilore_unit_exposure_risk with its partials in the library's fixed device
    array (no workspace): for callers that cannot allocate."""
    arr, n = _desc_array(units)
    _check("hilore_unit_exposure_risk_noalloc",
           load().hilore_unit_exposure_risk_noalloc(_p(coeff), _p(mask), int(rows), arr, n,
                                                    float(eps_alpha), float(eps_rel),
                                                    _p(exposure), _p(risk), _p(rel_err),
                                                    _stream(stream)))


def hilore_dequant_wgrad(x_codes, x_scales, code, block: int, dy, dw, K: int, M: int, N: int,
                         accumulate: bool = False, stream=None):
    _check("hilore_dequant_wgrad",
           load().hilore_dequant_wgrad(_p(x_codes), _p(x_scales), _code(code), int(block),
                                       _p(dy), _p(dw), int(K), int(M), int(N),
                                       1 if accumulate else 0, _stream(stream)))


def hilore_lora_grad_workspace_bytes(K: int, M: int, r: int) -> int:
    return int(load().hilore_lora_grad_workspace_bytes(int(K), int(M), int(r)))


def hilore_dequant_lora_grad(x_codes, x_scales, code, block: int, dh, da, K: int, M: int, r: int,
                             scale: float, accumulate: bool, workspace, stream=None):
    """dA [r, M] (+)= scale * dh^T xhat, xhat reconstructed from the codes in the
    operand load; dh bf16 [K, r]; workspace a device tensor of at least
    hilore_lora_grad_workspace_bytes(K, M, r) bytes."""
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("hilore_dequant_lora_grad",
           load().hilore_dequant_lora_grad(_p(x_codes), _p(x_scales), _code(code), int(block),
                                           _p(dh), _p(da), int(K), int(M), int(r), float(scale),
                                           1 if accumulate else 0, _p(workspace), ws_bytes,
                                           _stream(stream)))


def hilore_dequant_swiglu_bwd(gate: hilore_unit_desc, up: hilore_unit_desc, code, block: int, dh,
                              dgate, dup, stream=None):
    """dgate, dup (bf16 device tensors) from the gradient dh of h = silu(g) * u; each
    of gate / up is a unit descriptor: codes (+ scales) for an L operand, x for bf16."""
    _check("hilore_dequant_swiglu_bwd",
           load().hilore_dequant_swiglu_bwd(ctypes.byref(gate), ctypes.byref(up), _code(code),
                                            int(block), _p(dh), _p(dgate), _p(dup),
                                            _stream(stream)))


ACT_R, ACT_H, ACT_L = 0, 1, 2


def hilore_allocate_workspace_bytes(n_units: int, n_b: int = _d.N_B, n_d: int = _d.N_DELTA) -> int:
    return int(load().hilore_allocate_workspace_bytes(int(n_units), int(n_b), int(n_d)))


def hilore_allocate(q, verified, tau_h, tau_l, dm_h, dm_l, psi, m_res: float, delta_b: float,
                    n_b: int, n_d: int, action, totals, jk, workspace, stream=None):
    """Per-unit inputs and the outputs are device tensors (q, verified, action
    uint8; tau/dm/psi and totals float64; jk int64); workspace is a device
    tensor of at least hilore_allocate_workspace_bytes(...) bytes."""
    n = int(q.numel())
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("hilore_allocate",
           load().hilore_allocate(n, _p(q), _p(verified), _p(tau_h), _p(tau_l), _p(dm_h),
                                  _p(dm_l), _p(psi), float(m_res), float(delta_b), int(n_b),
                                  int(n_d), _p(action), _p(totals), _p(jk), _p(workspace),
                                  ws_bytes, _stream(stream)))


def hilore_grad_rel_err_workspace_bytes(n: int) -> int:
    return int(load().hilore_grad_rel_err_workspace_bytes(int(n)))


def hilore_grad_rel_err(g_l, g_ex, y, workspace, eps_num: float = _d.EPS_NUM, stream=None):
    """y (a one-element f32 device tensor or view) = relative gradient error of
    g_l against g_ex (f32 device tensors of equal size)."""
    n = int(g_ex.numel())
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("hilore_grad_rel_err",
           load().hilore_grad_rel_err(_p(g_l), _p(g_ex), n, float(eps_num), _p(y), _p(workspace),
                                      ws_bytes, _stream(stream)))


def hilore_calibrate(unit_class, exposure, rel_err, grad_err, n_classes: int, kappa, ebar,
                     stream=None):
    """exposure, rel_err, grad_err: f32 device tensors [n_batches, n_units];
    unit_class i32 [n_units]; kappa f64 [n_classes], ebar f64 [n_units]."""
    nb, nu = (int(d) for d in exposure.shape)
    _check("hilore_calibrate",
           load().hilore_calibrate(nu, nb, int(n_classes), _p(unit_class), _p(exposure),
                                   _p(rel_err), _p(grad_err), _p(kappa), _p(ebar),
                                   _stream(stream)))


def hilore_risk_score(unit_class, kappa, ebar, exposure, psi, stream=None):
    _check("hilore_risk_score",
           load().hilore_risk_score(int(unit_class.numel()), _p(unit_class), int(kappa.numel()),
                                    _p(kappa), _p(ebar), _p(exposure), _p(psi), _stream(stream)))


def hilore_update_sparsity(coeff, flags, adv, mask, R: int, T: int, top_frac: float, counts,
                           top_share, stream=None):
    _check("hilore_update_sparsity",
           load().hilore_update_sparsity(_p(coeff), _p(flags), _p(adv), _p(mask), int(R), int(T),
                                         float(top_frac), _p(counts), _p(top_share),
                                         _stream(stream)))
