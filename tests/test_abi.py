"""The C-ABI library on the host: it loads, exports every entry point that
include/hilore.h declares, and rejects invalid arguments before touching the
device (so these checks run without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_2609_33570_amd import hilore

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hilore.h")

# A fake but 16-byte aligned "device" address: never dereferenced, because
# every call below fails validation first.
FAKE = 1 << 20


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(hilore.LIB_PATH):
        from paper_2609_33570_amd import _build

        _build.build()
    return hilore.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hilore_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert {"hilore_grpo_coeffs", "hilore_compress", "hilore_decompress",
            "hilore_unit_exposure_risk", "hilore_dequant_wgrad"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_version(lib):
    assert hilore.status_string(0) == "HILORE_OK"
    assert hilore.status_string(3) == "HILORE_ERR_UNSUPPORTED"
    assert hilore.status_string(99) == "HILORE_ERR_UNKNOWN"
    assert hilore.version() >= 10000


def grpo(lib, **kw):
    a = dict(rewards=FAKE, logp_new=FAKE, logp_old=FAKE, logp_ref=None, mask=None, P=2, G=8,
             T=16, clip_eps=0.2, adv_eps=1e-6, beta=0.0, n_norm=0.0, adv=FAKE, ratio=None,
             flags=FAKE, coeff=FAKE, ws=None, ws_bytes=0)
    a.update(kw)
    return lib.hilore_grpo_coeffs(a["rewards"], a["logp_new"], a["logp_old"], a["logp_ref"],
                                  a["mask"], a["P"], a["G"], a["T"], a["clip_eps"],
                                  a["adv_eps"], a["beta"], a["n_norm"], a["adv"], a["ratio"],
                                  a["flags"], a["coeff"], a["ws"], a["ws_bytes"], None)


def test_grpo_validation(lib):
    assert grpo(lib, G=65) == hilore.HILORE_ERR_UNSUPPORTED
    assert grpo(lib, G=0) == hilore.HILORE_ERR_INVALID_ARG
    assert grpo(lib, P=-1) == hilore.HILORE_ERR_INVALID_ARG
    assert grpo(lib, T=-1) == hilore.HILORE_ERR_INVALID_ARG
    assert grpo(lib, P=1 << 20, G=64, T=1 << 12) == hilore.HILORE_ERR_UNSUPPORTED
    assert grpo(lib, clip_eps=0.0) == hilore.HILORE_ERR_INVALID_ARG
    assert grpo(lib, clip_eps=1.0) == hilore.HILORE_ERR_INVALID_ARG
    assert grpo(lib, beta=-1.0) == hilore.HILORE_ERR_INVALID_ARG
    assert grpo(lib, beta=1e-3) == hilore.HILORE_ERR_INVALID_ARG  # logp_ref missing
    assert grpo(lib, rewards=None) == hilore.HILORE_ERR_INVALID_ARG
    assert grpo(lib, coeff=None) == hilore.HILORE_ERR_INVALID_ARG
    assert grpo(lib, flags=None) == hilore.HILORE_ERR_INVALID_ARG
    assert grpo(lib, logp_new=FAKE + 4) == hilore.HILORE_ERR_ALIGNMENT
    assert grpo(lib, mask=FAKE + 8) == hilore.HILORE_ERR_ALIGNMENT


def test_grpo_workspace(lib):
    """N counted over more than 2^16 slots needs the pre-pass workspace: 4 bytes
    per 2^16 slots, at most 1 KB; nothing for smaller calls or a given N."""
    f = lib.hilore_grpo_coeffs_workspace_bytes
    assert f(1, 8, 2048) == 0 and f(2, 16, 2048) == 0          # 16384 and 65536 slots
    assert f(2, 16, 2049) == 2 * 4                             # just above 2^16
    assert f(2, 16, 1 << 21) == 256 * 4 and f(64, 64, 1 << 18) == 256 * 4
    assert f(-1, 8, 16) == 0 and f(1, 0, 16) == 0
    big = dict(P=16, G=16, T=1024, mask=FAKE)                  # 2^18 slots
    assert grpo(lib, **big) == hilore.HILORE_ERR_INVALID_ARG   # no workspace
    assert grpo(lib, ws=FAKE, ws_bytes=15, **big) == hilore.HILORE_ERR_WORKSPACE
    assert grpo(lib, ws=FAKE + 4, ws_bytes=16, **big) == hilore.HILORE_ERR_ALIGNMENT
    assert grpo(lib, P=0) == hilore.HILORE_OK  # nothing to do, nothing launched


def unit(**kw):
    d = dict(x=FAKE, codes=FAKE, scales=FAKE, xhat=FAKE, row_ss_x=None, row_ss_err=None,
             rows=4, cols=256, ld=256)
    d.update(kw)
    return hilore.hilore_unit_desc(d["x"], d["codes"], d["scales"], d["xhat"], d["row_ss_x"],
                                   d["row_ss_err"], d["rows"], d["cols"], d["ld"])


def codec(lib, fn, units, code=0, block=128):
    arr = (hilore.hilore_unit_desc * max(1, len(units)))(*units)
    return getattr(lib, fn)(arr, len(units), code, block, None)


@pytest.mark.parametrize("fn", ["hilore_compress", "hilore_decompress"])
def test_codec_validation(lib, fn):
    E = hilore
    assert codec(lib, fn, [unit()], code=3) == E.HILORE_ERR_INVALID_ARG
    # the literal cast has no blocks: block must be 0, and scales are not needed
    assert codec(lib, fn, [unit()], code=2) == E.HILORE_ERR_INVALID_ARG
    assert codec(lib, fn, [unit(scales=None, codes=FAKE + 1)], code=2, block=0) == E.HILORE_ERR_ALIGNMENT
    assert codec(lib, fn, [unit(scales=None, codes=None)], code=2, block=0) == E.HILORE_ERR_INVALID_ARG
    assert codec(lib, fn, [unit()], block=48) == E.HILORE_ERR_UNSUPPORTED
    assert codec(lib, fn, [unit()], block=512) == E.HILORE_ERR_UNSUPPORTED
    assert codec(lib, fn, [unit(cols=200)], block=128) == E.HILORE_ERR_UNSUPPORTED
    assert codec(lib, fn, [unit(rows=-1)]) == E.HILORE_ERR_INVALID_ARG
    assert codec(lib, fn, [unit(codes=None)]) == E.HILORE_ERR_INVALID_ARG
    assert codec(lib, fn, [unit(scales=None)]) == E.HILORE_ERR_INVALID_ARG
    assert codec(lib, fn, [unit(scales=FAKE + 4)]) == E.HILORE_ERR_ALIGNMENT
    # a bad unit anywhere in the list rejects the whole call
    assert codec(lib, fn, [unit()] * 20 + [unit(codes=None)]) == E.HILORE_ERR_INVALID_ARG
    assert getattr(lib, fn)(None, 1, 0, 128, None) == E.HILORE_ERR_INVALID_ARG
    assert getattr(lib, fn)(None, -1, 0, 128, None) == E.HILORE_ERR_INVALID_ARG
    assert getattr(lib, fn)(None, 0, 0, 128, None) == E.HILORE_OK
    # empty units are skipped without a launch
    assert codec(lib, fn, [unit(rows=0, codes=None, x=None, xhat=None)]) == E.HILORE_OK
    # row lengths beyond 2^30 (32-bit in-row byte offsets) and more than 2^30 rows
    big = (1 << 30) + 128
    assert codec(lib, fn, [unit(cols=big, ld=big)]) == E.HILORE_ERR_UNSUPPORTED
    assert codec(lib, fn, [unit(rows=(1 << 30) + 1)]) == E.HILORE_ERR_UNSUPPORTED


def test_compress_specific_validation(lib):
    E = hilore
    f = "hilore_compress"
    assert codec(lib, f, [unit(x=None)]) == E.HILORE_ERR_INVALID_ARG
    assert codec(lib, f, [unit(ld=128)]) == E.HILORE_ERR_INVALID_ARG
    assert codec(lib, f, [unit(ld=260)]) == E.HILORE_ERR_ALIGNMENT
    assert codec(lib, f, [unit(x=FAKE + 2)]) == E.HILORE_ERR_ALIGNMENT
    assert codec(lib, f, [unit(row_ss_x=FAKE + 4)]) == E.HILORE_ERR_ALIGNMENT


def test_decompress_specific_validation(lib):
    assert codec(lib, "hilore_decompress", [unit(xhat=None)]) == hilore.HILORE_ERR_INVALID_ARG


def risk(lib, units, rows=4, coeff=FAKE, mask=None, outs=(FAKE, FAKE, FAKE), eps=(1e-8, 1e-8),
         ws=FAKE, ws_bytes=1 << 20):
    arr = (hilore.hilore_unit_desc * max(1, len(units)))(*units)
    return lib.hilore_unit_exposure_risk(coeff, mask, rows, arr, len(units), eps[0], eps[1],
                                         outs[0], outs[1], outs[2], ws, ws_bytes, None)


def test_exposure_risk_validation(lib):
    E = hilore
    ok = unit(row_ss_x=FAKE, row_ss_err=FAKE)
    assert risk(lib, [unit()]) == E.HILORE_ERR_INVALID_ARG          # row sums missing
    assert risk(lib, [ok], rows=5) == E.HILORE_ERR_INVALID_ARG      # rows disagree
    assert risk(lib, [ok], coeff=None) == E.HILORE_ERR_INVALID_ARG
    assert risk(lib, [ok], outs=(None, FAKE, FAKE)) == E.HILORE_ERR_INVALID_ARG
    assert risk(lib, [ok], mask=FAKE + 1) == E.HILORE_ERR_ALIGNMENT
    assert risk(lib, [ok], outs=(FAKE, FAKE + 2, FAKE)) == E.HILORE_ERR_ALIGNMENT
    assert risk(lib, [ok], eps=(-1.0, 1e-8)) == E.HILORE_ERR_INVALID_ARG
    assert risk(lib, [unit(row_ss_x=FAKE, row_ss_err=FAKE, cols=0)]) == E.HILORE_ERR_INVALID_ARG
    assert risk(lib, []) == E.HILORE_OK
    assert risk(lib, [ok], ws=None) == E.HILORE_ERR_INVALID_ARG
    assert risk(lib, [ok], ws=FAKE + 8) == E.HILORE_ERR_ALIGNMENT
    assert risk(lib, [ok], ws_bytes=31) == E.HILORE_ERR_WORKSPACE
    big = unit(row_ss_x=FAKE, row_ss_err=FAKE, rows=1 << 24)
    assert risk(lib, [big], rows=1 << 24) == E.HILORE_ERR_UNSUPPORTED


def test_exposure_risk_workspace_size(lib):
    """32 bytes per unit per chunk of 2048 rows; nothing without rows."""
    f = lib.hilore_unit_exposure_risk_workspace_bytes
    assert f(16384, 2) == 2 * 8 * 32
    assert f(16384, 78) == 78 * 8 * 32
    assert f(2049, 3) == 3 * 2 * 32
    assert f(1, 1) == 32 and f(0, 5) == 0 and f(100, 0) == 0
    assert f(-1, 1) == 0 and f(1 << 24, 1) == 0


def wgrad(lib, **kw):
    a = dict(x_codes=FAKE, x_scales=FAKE, code=1, block=128, dy=FAKE, dw=FAKE, K=256, M=512,
             N=512, accumulate=0)
    a.update(kw)
    return lib.hilore_dequant_wgrad(a["x_codes"], a["x_scales"], a["code"], a["block"], a["dy"],
                                    a["dw"], a["K"], a["M"], a["N"], a["accumulate"], None)


def test_wgrad_validation(lib):
    E = hilore
    assert wgrad(lib, M=192) == E.HILORE_ERR_UNSUPPORTED        # M % block
    assert wgrad(lib, N=100) == E.HILORE_ERR_UNSUPPORTED        # N % 8
    assert wgrad(lib, block=100) == E.HILORE_ERR_UNSUPPORTED
    assert wgrad(lib, code=7) == E.HILORE_ERR_INVALID_ARG
    assert wgrad(lib, K=-1) == E.HILORE_ERR_INVALID_ARG
    assert wgrad(lib, dw=None) == E.HILORE_ERR_INVALID_ARG
    assert wgrad(lib, dy=None) == E.HILORE_ERR_INVALID_ARG
    assert wgrad(lib, x_scales=FAKE + 4) == E.HILORE_ERR_ALIGNMENT
    assert wgrad(lib, M=0) == E.HILORE_OK
    assert wgrad(lib, M=1 << 22) == E.HILORE_ERR_UNSUPPORTED    # M, N below 2^22
    assert wgrad(lib, N=1 << 22) == E.HILORE_ERR_UNSUPPORTED
    # the literal cast: block 0 only, no M % block rule, scales may be NULL
    assert wgrad(lib, code=2) == E.HILORE_ERR_INVALID_ARG
    assert wgrad(lib, code=2, block=0, N=100) == E.HILORE_ERR_UNSUPPORTED
    assert wgrad(lib, code=2, block=0, x_scales=None, x_codes=FAKE + 1) == E.HILORE_ERR_ALIGNMENT
    assert wgrad(lib, code=2, block=0, x_scales=None, dy=None) == E.HILORE_ERR_INVALID_ARG


def alloc(lib, **kw):
    a = dict(U=4, q=FAKE, verified=FAKE, tau_h=FAKE, tau_l=FAKE, dm_h=FAKE, dm_l=FAKE, psi=FAKE,
             m_res=1.0, delta_b=1.0, n_b=1024, n_d=1024, action=FAKE, totals=FAKE, jk=FAKE,
             ws=FAKE, ws_bytes=None)
    a.update(kw)
    if a["ws_bytes"] is None:
        a["ws_bytes"] = lib.hilore_allocate_workspace_bytes(a["U"], a["n_b"], a["n_d"]) - 1
    return lib.hilore_allocate(a["U"], a["q"], a["verified"], a["tau_h"], a["tau_l"], a["dm_h"],
                               a["dm_l"], a["psi"], a["m_res"], a["delta_b"], a["n_b"], a["n_d"],
                               a["action"], a["totals"], a["jk"], a["ws"], a["ws_bytes"], None)


def test_allocate_workspace_size(lib):
    f = lib.hilore_allocate_workspace_bytes
    one = f(1, 1024, 1024)
    # two fp64 tables of 1025 rows x 1088 padded cells, and 2 bits per cell per unit
    assert one >= 2 * 8 * 1025 * 1088 + 1025 * 1088 // 4
    assert abs(f(11, 1024, 1024) - one - 10 * 1025 * 1088 // 4) < 256
    assert f(0, 1, 1) > 0
    assert f(-1, 1024, 1024) == 0 and f(1, 0, 1024) == 0 and f(1, 4097, 1024) == 0


def test_allocate_validation(lib):
    E = hilore
    big = 1 << 40
    # a workspace one byte short of what is needed
    assert alloc(lib) == E.HILORE_ERR_WORKSPACE
    assert alloc(lib, U=-1, ws_bytes=big) == E.HILORE_ERR_INVALID_ARG
    assert alloc(lib, n_b=0, ws_bytes=big) == E.HILORE_ERR_INVALID_ARG
    assert alloc(lib, n_d=0, ws_bytes=big) == E.HILORE_ERR_INVALID_ARG
    assert alloc(lib, n_b=4097, ws_bytes=big) == E.HILORE_ERR_UNSUPPORTED
    assert alloc(lib, m_res=-1.0, ws_bytes=big) == E.HILORE_ERR_INVALID_ARG
    assert alloc(lib, delta_b=float("inf"), ws_bytes=big) == E.HILORE_ERR_INVALID_ARG
    assert alloc(lib, delta_b=float("nan"), ws_bytes=big) == E.HILORE_ERR_INVALID_ARG
    for name in ("q", "verified", "tau_h", "tau_l", "dm_h", "dm_l", "psi", "action", "totals",
                 "jk", "ws"):
        assert alloc(lib, ws_bytes=big, **{name: None}) == E.HILORE_ERR_INVALID_ARG, name
    for name in ("tau_h", "psi", "totals", "jk"):
        assert alloc(lib, ws_bytes=big, **{name: FAKE + 4}) == E.HILORE_ERR_ALIGNMENT, name
    assert alloc(lib, ws_bytes=big, ws=FAKE + 8) == E.HILORE_ERR_ALIGNMENT
    # per-unit arrays are not needed without units, but the outputs still are
    assert alloc(lib, U=0, q=None, tau_h=None, totals=None, ws_bytes=big) == \
        E.HILORE_ERR_INVALID_ARG
    # zero budgets leave a single state per axis: a small workspace is checked too
    assert alloc(lib, m_res=0.0, delta_b=0.0, ws_bytes=1000) == E.HILORE_ERR_WORKSPACE


def test_calibration_entry_points_validate(lib):
    E = hilore
    big = 1 << 20
    ws = lib.hilore_grad_rel_err_workspace_bytes
    assert ws(0) == 16 and ws(1 << 20) == 256 * 16 and ws(1 << 24) == 1024 * 16 and ws(1 << 30) == 1024 * 16 and ws(-1) == 0
    rel = lib.hilore_grad_rel_err
    assert rel(FAKE, FAKE, 1000, 1e-30, FAKE, FAKE, 15, None) == E.HILORE_ERR_WORKSPACE
    assert rel(FAKE, FAKE, -1, 1e-30, FAKE, FAKE, big, None) == E.HILORE_ERR_INVALID_ARG
    assert rel(FAKE, FAKE, 10, 0.0, FAKE, FAKE, big, None) == E.HILORE_ERR_INVALID_ARG
    assert rel(FAKE, FAKE, 10, float("inf"), FAKE, FAKE, big, None) == E.HILORE_ERR_INVALID_ARG
    assert rel(None, FAKE, 10, 1e-30, FAKE, FAKE, big, None) == E.HILORE_ERR_INVALID_ARG
    assert rel(FAKE, FAKE, 10, 1e-30, None, FAKE, big, None) == E.HILORE_ERR_INVALID_ARG
    assert rel(FAKE + 4, FAKE, 10, 1e-30, FAKE, FAKE, big, None) == E.HILORE_ERR_ALIGNMENT
    assert rel(FAKE, FAKE, 10, 1e-30, FAKE + 2, FAKE, big, None) == E.HILORE_ERR_ALIGNMENT
    assert rel(FAKE, FAKE, 10, 1e-30, FAKE, FAKE + 8, big, None) == E.HILORE_ERR_ALIGNMENT

    cal = lib.hilore_calibrate
    assert cal(-1, 2, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == E.HILORE_ERR_INVALID_ARG
    assert cal(4, 2, -1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == E.HILORE_ERR_INVALID_ARG
    assert cal(1 << 16, 1 << 15, 1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == \
        E.HILORE_ERR_UNSUPPORTED
    assert cal(4, 2, 1, FAKE, None, FAKE, FAKE, FAKE, FAKE, None) == E.HILORE_ERR_INVALID_ARG
    assert cal(4, 2, 1, FAKE, FAKE, FAKE, FAKE, None, FAKE, None) == E.HILORE_ERR_INVALID_ARG
    assert cal(4, 2, 1, FAKE, FAKE, FAKE + 2, FAKE, FAKE, FAKE, None) == E.HILORE_ERR_ALIGNMENT
    assert cal(4, 2, 1, FAKE, FAKE, FAKE, FAKE, FAKE + 4, FAKE, None) == E.HILORE_ERR_ALIGNMENT

    risk = lib.hilore_risk_score
    assert risk(-1, FAKE, 1, FAKE, FAKE, FAKE, FAKE, None) == E.HILORE_ERR_INVALID_ARG
    assert risk(4, FAKE, 1, FAKE, FAKE, FAKE, None, None) == E.HILORE_ERR_INVALID_ARG
    assert risk(4, FAKE, 1, FAKE, FAKE, FAKE, FAKE + 4, None) == E.HILORE_ERR_ALIGNMENT
    assert risk(0, None, 0, None, None, None, None, None) == E.HILORE_OK

    sp = lib.hilore_update_sparsity
    assert sp(FAKE, FAKE, FAKE, None, 4, 8, 0.0, FAKE, FAKE, None) == E.HILORE_ERR_INVALID_ARG
    assert sp(FAKE, FAKE, FAKE, None, 4, 8, 1.5, FAKE, FAKE, None) == E.HILORE_ERR_INVALID_ARG
    assert sp(FAKE, FAKE, FAKE, None, -4, 8, 0.1, FAKE, FAKE, None) == E.HILORE_ERR_INVALID_ARG
    assert sp(FAKE, FAKE, FAKE, None, 1 << 16, 1 << 15, 0.1, FAKE, FAKE, None) == \
        E.HILORE_ERR_UNSUPPORTED
    assert sp(FAKE, None, FAKE, None, 4, 8, 0.1, FAKE, FAKE, None) == E.HILORE_ERR_INVALID_ARG
    assert sp(FAKE, FAKE, FAKE, None, 4, 8, 0.1, None, FAKE, None) == E.HILORE_ERR_INVALID_ARG
    assert sp(FAKE, FAKE, FAKE, None, 4, 8, 0.1, FAKE + 4, FAKE, None) == E.HILORE_ERR_ALIGNMENT


def test_lora_grad_validation(lib):
    E = hilore
    ws = lib.hilore_lora_grad_workspace_bytes
    # 256 workgroups x 2 partial [16 R][256] fp32 slots (a range meets at most two
    # strips), R = row blocks of 16 in the widest pass (passes of up to 80 rows)
    assert ws(16384, 18944, 16) == 256 * 2 * 16 * 256 * 4
    assert ws(16384, 18944, 64) == 4 * ws(16384, 18944, 16)
    assert ws(16384, 18944, 80) == 5 * ws(16384, 18944, 16)
    assert ws(16384, 18944, 96) == ws(16384, 18944, 80)  # later passes reuse the slots
    assert ws(16384, 18944, 18) == 2 * ws(16384, 18944, 16)
    assert ws(32, 256, 16) == 1 * 2 * 16 * 256 * 4       # one k-step: one workgroup
    assert ws(-1, 256, 16) == 0 and ws(32, 256, 0) == 0
    big = 1 << 30

    def call(**kw):
        a = dict(codes=FAKE, scales=FAKE, code=1, block=128, dh=FAKE, da=FAKE, K=1024, M=1024,
                 r=16, scale=2.0, acc=0, ws=FAKE, ws_bytes=big)
        a.update(kw)
        return lib.hilore_dequant_lora_grad(a["codes"], a["scales"], a["code"], a["block"],
                                            a["dh"], a["da"], a["K"], a["M"], a["r"], a["scale"],
                                            a["acc"], a["ws"], a["ws_bytes"], None)
    assert call(ws_bytes=ws(1024, 1024, 16) - 1) == E.HILORE_ERR_WORKSPACE
    assert call(K=-1) == E.HILORE_ERR_INVALID_ARG
    assert call(r=0) == E.HILORE_ERR_INVALID_ARG
    assert call(scale=float("nan")) == E.HILORE_ERR_INVALID_ARG
    assert call(code=7) == E.HILORE_ERR_INVALID_ARG
    assert call(block=48) == E.HILORE_ERR_UNSUPPORTED
    assert call(M=1000) == E.HILORE_ERR_UNSUPPORTED            # not a block multiple
    assert call(code=2, block=0, M=1000) == E.HILORE_ERR_UNSUPPORTED  # not a multiple of 16
    assert call(r=4098) == E.HILORE_ERR_UNSUPPORTED
    assert call(r=17) == E.HILORE_ERR_UNSUPPORTED  # odd ranks: dh rows are read in pairs
    for name in ("codes", "scales", "dh", "da", "ws"):
        assert call(**{name: None}) == E.HILORE_ERR_INVALID_ARG, name
    for name in ("codes", "scales", "dh", "da", "ws"):
        assert call(**{name: FAKE + 8}) == E.HILORE_ERR_ALIGNMENT, name
    assert call(M=0, da=None) == E.HILORE_OK  # nothing to do


def test_swiglu_bwd_validation(lib):
    E = hilore

    def desc(**kw):
        d = dict(x=FAKE, codes=None, scales=None, xhat=None, row_ss_x=None, row_ss_err=None,
                 rows=64, cols=256, ld=256)
        d.update(kw)
        return hilore.hilore_unit_desc(d["x"], d["codes"], d["scales"], d["xhat"], d["row_ss_x"],
                                       d["row_ss_err"], d["rows"], d["cols"], d["ld"])

    def call(g=None, u=None, code=1, block=128, dh=FAKE, dg=FAKE, du=FAKE):
        g = g if g is not None else desc(x=None, codes=FAKE, scales=FAKE)
        u = u if u is not None else desc()
        return lib.hilore_dequant_swiglu_bwd(ctypes.byref(g), ctypes.byref(u), code, block, dh,
                                             dg, du, None)
    assert lib.hilore_dequant_swiglu_bwd(None, ctypes.byref(desc()), 1, 128, FAKE, FAKE, FAKE,
                                         None) == E.HILORE_ERR_INVALID_ARG
    assert call(u=desc(rows=63)) == E.HILORE_ERR_INVALID_ARG
    assert call(u=desc(cols=248, ld=256), g=desc(x=None, codes=FAKE, scales=FAKE, cols=248)) == \
        E.HILORE_ERR_UNSUPPORTED  # cols not a block multiple
    assert call(g=desc(cols=252, ld=256), u=desc(cols=252, ld=256)) == E.HILORE_ERR_UNSUPPORTED
    assert call(code=9) == E.HILORE_ERR_INVALID_ARG
    assert call(block=48) == E.HILORE_ERR_UNSUPPORTED
    assert call(g=desc(x=None, codes=FAKE, scales=None)) == E.HILORE_ERR_INVALID_ARG
    assert call(u=desc(x=None)) == E.HILORE_ERR_INVALID_ARG
    assert call(u=desc(ld=200)) == E.HILORE_ERR_INVALID_ARG
    assert call(u=desc(ld=260)) == E.HILORE_ERR_ALIGNMENT
    assert call(u=desc(x=FAKE + 4)) == E.HILORE_ERR_ALIGNMENT
    assert call(g=desc(x=None, codes=FAKE + 8, scales=FAKE)) == E.HILORE_ERR_ALIGNMENT
    assert call(dh=None) == E.HILORE_ERR_INVALID_ARG
    assert call(du=FAKE + 2) == E.HILORE_ERR_ALIGNMENT
    assert call(g=desc(x=None, codes=FAKE, scales=FAKE, rows=0), u=desc(rows=0)) == E.HILORE_OK


class _FakeDeviceTensor:
    """Just enough of a device tensor for the binding's marshalling checks."""

    def __init__(self, shape, strides, contiguous):
        self.is_cuda, self.shape, self._strides, self._contig = True, shape, strides, contiguous
        self.device = "cuda:0"

    def is_contiguous(self):
        return self._contig

    def stride(self, dim=None):
        return self._strides if dim is None else self._strides[dim]

    def dim(self):
        return len(self.shape)

    def data_ptr(self):
        return FAKE


def test_binding_refuses_host_and_strided_tensors(lib):
    """A host tensor would give the kernels a host address, a strided view the
    wrong elements: the binding refuses both before anything reaches the
    library."""
    import torch
    x = torch.zeros(4, 8, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="device"):
        hilore.unit_desc(x=x)
    with pytest.raises(ValueError, match="device"):
        hilore.hilore_grad_rel_err(torch.zeros(4), torch.zeros(4), torch.zeros(1),
                                   torch.zeros(2, dtype=torch.float64))
    with pytest.raises(ValueError, match="dense"):
        hilore._p(_FakeDeviceTensor((4, 8), (1, 4), False))  # a transposed view
    assert hilore._p(_FakeDeviceTensor((4, 8), (8, 1), True)) == FAKE
    # a unit's x may have padded rows, not strided columns
    assert hilore._p_rows(_FakeDeviceTensor((4, 8), (16, 1), False)) == FAKE
    with pytest.raises(ValueError, match="contiguous rows"):
        hilore._p_rows(_FakeDeviceTensor((4, 8), (1, 4), False))
