"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every entry point that include/roi.h declares, and rejects invalid arguments
on the host before anything is launched."""
from __future__ import annotations

import ctypes
import math
import os
import re

import pytest

import paper_2608_23048_amd as roi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "roi.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(roi_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(roi.LIB_PATH):
        pytest.fail("libroi.so is not built (run __graft_entry__.build())")
    return roi.lib()


def test_exports_every_declared_symbol(L):
    names = header_functions()
    assert {"roi_mask_fwd", "roi_mask_fwd_soft", "roi_mask_bwd", "roi_gumbel_noise",
            "roi_gumbel_from_words", "roi_fast_noise_from_words",
            "roi_mask_fwd_grouped", "roi_mask_fwd_soft_grouped", "roi_mask_bwd_grouped",
            "roi_mask_bwd_adamw", "roi_mask_bwd_adamw_grouped", "roi_mask_export",
            "roi_cat_num_candidates", "roi_cat_mask_fwd", "roi_cat_mask_bwd",
            "roi_anneal", "roi_status_string", "roi_last_error", "roi_abi_version"} <= set(names)
    for name in names:
        assert hasattr(L, name), name


def test_version_and_status_strings(L):
    assert L.roi_abi_version() == 1
    for st in (roi.ROI_OK, roi.ROI_E_INVAL, roi.ROI_E_UNSUPPORTED, roi.ROI_E_HIP):
        assert L.roi_status_string(st)
    assert L.roi_status_string(12345) == b"unknown status"


FAKE = 0x7F0000000000  # 16-byte aligned, never dereferenced: every call below fails validation


def fwd(L, **kw):
    a = dict(W=FAKE, logits=FAKE + (1 << 30), rows=4, cols=8, n=2, m=4, tau=1.0, lam=1.0, seed=0,
             step=0, off=0, Wm=FAKE + (2 << 30), S=None, idx=None)
    a.update(kw)
    return L.roi_mask_fwd(a["W"], a["logits"], a["rows"], a["cols"], a["n"], a["m"], a["tau"],
                          a["lam"], a["seed"], a["step"], a["off"], a["Wm"], a["S"], a["idx"], None)


def bwd(L, **kw):
    a = dict(G=FAKE, W=FAKE + (1 << 30), logits=FAKE + (2 << 30), rows=4, cols=8, n=2, m=4,
             tau=1.0, lam=1.0, seed=0, step=0, off=0, d=FAKE + (3 << 30))
    a.update(kw)
    return L.roi_mask_bwd(a["G"], a["W"], a["logits"], a["rows"], a["cols"], a["n"], a["m"],
                          a["tau"], a["lam"], a["seed"], a["step"], a["off"], a["d"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(n=0), roi.ROI_E_INVAL),
    (dict(n=5), roi.ROI_E_INVAL),
    (dict(m=3, n=1, cols=9), roi.ROI_E_UNSUPPORTED),
    (dict(m=12, n=6, cols=12), roi.ROI_E_UNSUPPORTED),
    (dict(m=64, n=32, cols=64), roi.ROI_E_UNSUPPORTED),
    (dict(cols=6), roi.ROI_E_INVAL),
    (dict(rows=-1), roi.ROI_E_INVAL),
    (dict(rows=1 << 40, cols=1 << 40), roi.ROI_E_INVAL),
    (dict(tau=0.0), roi.ROI_E_INVAL),
    (dict(tau=-1.0), roi.ROI_E_INVAL),
    (dict(tau=math.inf), roi.ROI_E_INVAL),
    (dict(tau=math.nan), roi.ROI_E_INVAL),
    (dict(lam=0.0), roi.ROI_E_INVAL),
    (dict(lam=math.nan), roi.ROI_E_INVAL),
    (dict(off=2), roi.ROI_E_INVAL),
    (dict(off=4, m=8, n=4), roi.ROI_E_INVAL),
    (dict(off=2**64 - 4), roi.ROI_E_INVAL),
    (dict(W=None), roi.ROI_E_INVAL),
    (dict(Wm=None), roi.ROI_E_INVAL),
    (dict(W=FAKE + 8), roi.ROI_E_INVAL),
    (dict(S=FAKE + (3 << 30) + 4), roi.ROI_E_INVAL),
    (dict(Wm=FAKE + 16), roi.ROI_E_INVAL),              # overlaps W
    (dict(S=FAKE + (1 << 30) + 16), roi.ROI_E_INVAL),   # overlaps logits
    (dict(idx=FAKE + (2 << 30) + 32), roi.ROI_E_INVAL),  # overlaps W_masked
])
def test_fwd_rejects_before_launch(L, kw, status):
    assert fwd(L, **kw) == status
    assert L.roi_last_error()
    a = dict(W=FAKE, logits=FAKE + (1 << 30), rows=4, cols=8, n=2, m=4, tau=1.0, lam=1.0, seed=0,
             step=0, off=0, Wm=FAKE + (2 << 30), S=None, idx=None)
    a.update(kw)
    assert L.roi_mask_fwd_soft(a["W"], a["logits"], a["rows"], a["cols"], a["n"], a["m"],
                               a["tau"], a["lam"], a["seed"], a["step"], a["off"], a["Wm"],
                               a["S"], a["idx"], None) == status


@pytest.mark.parametrize("kw,status", [
    (dict(n=0), roi.ROI_E_INVAL),
    (dict(m=64, n=16, cols=64), roi.ROI_E_UNSUPPORTED),
    (dict(m=16, n=8, cols=24), roi.ROI_E_INVAL),
    (dict(cols=10), roi.ROI_E_INVAL),
    (dict(tau=0.0), roi.ROI_E_INVAL),
    (dict(lam=-2.0), roi.ROI_E_INVAL),
    (dict(off=6), roi.ROI_E_INVAL),
    (dict(d=None), roi.ROI_E_INVAL),
    (dict(G=FAKE + 2), roi.ROI_E_INVAL),
    (dict(d=FAKE + (2 << 30)), roi.ROI_E_INVAL),  # aliases logits
])
def test_bwd_rejects_before_launch(L, kw, status):
    assert bwd(L, **kw) == status


GB = 1 << 30


def fwd_desc(i, **kw):
    """Fake descriptor i (disjoint 1 GiB slots per tensor); never launched."""
    base = FAKE + i * 8 * GB
    a = dict(W=base, logits=base + GB, W_masked=base + 2 * GB, soft_mask=None, sel_idx=None,
             rows=4, cols=8, elem_offset=i * 32)
    a.update(kw)
    return roi.FwdTensor(a["W"], a["logits"], a["W_masked"], a["soft_mask"], a["sel_idx"],
                         a["rows"], a["cols"], a["elem_offset"])


def bwd_desc(i, **kw):
    base = FAKE + i * 8 * GB
    a = dict(G=base, W=base + GB, logits=base + 2 * GB, d=base + 3 * GB, rows=4, cols=8,
             elem_offset=i * 32)
    a.update(kw)
    return roi.BwdTensor(a["G"], a["W"], a["logits"], a["d"], a["rows"], a["cols"],
                         a["elem_offset"])


def grouped(L, fn, descs, n=2, m=4, tau=1.0, lam=1.0):
    T = type(descs[0]) if descs else roi.FwdTensor
    arr = (T * max(1, len(descs)))(*descs)
    return getattr(L, fn)(ctypes.addressof(arr), len(descs), n, m, tau, lam, 0, 0, None)


@pytest.mark.parametrize("fn", ["roi_mask_fwd_grouped", "roi_mask_fwd_soft_grouped"])
def test_fwd_grouped_rejects_before_launch(L, fn):
    ok = [fwd_desc(0), fwd_desc(1)]
    cases = [
        ([ok[0], fwd_desc(1, cols=6)], roi.ROI_E_INVAL, "tensor 1"),
        ([ok[0], fwd_desc(1, elem_offset=34)], roi.ROI_E_INVAL, "tensor 1"),
        ([ok[0], fwd_desc(1, W=None)], roi.ROI_E_INVAL, "tensor 1"),
        ([fwd_desc(0, logits=FAKE + GB + 4), ok[1]], roi.ROI_E_INVAL, "tensor 0"),
        ([fwd_desc(0, sel_idx=FAKE + 3 * GB), ok[1]], roi.ROI_E_INVAL, "every tensor"),
        ([ok[0], fwd_desc(1, soft_mask=FAKE + 8 * GB + 3 * GB)], roi.ROI_E_INVAL, "every tensor"),
        ([ok[0], fwd_desc(1, W_masked=FAKE + GB + 64)], roi.ROI_E_INVAL, "overlap"),  # into logits 0
        ([ok[0], fwd_desc(1, W_masked=FAKE + 2 * GB)], roi.ROI_E_INVAL, "overlap"),  # same output
    ]
    for descs, status, msg in cases:
        assert grouped(L, fn, descs) == status
        assert msg in L.roi_last_error().decode()
    assert grouped(L, fn, ok, m=12, n=6) == roi.ROI_E_UNSUPPORTED
    assert grouped(L, fn, ok, tau=0.0) == roi.ROI_E_INVAL
    assert L.roi_mask_fwd_grouped(None, 2, 2, 4, 1.0, 1.0, 0, 0, None) == roi.ROI_E_INVAL
    assert L.roi_mask_fwd_grouped(None, -1, 2, 4, 1.0, 1.0, 0, 0, None) == roi.ROI_E_INVAL
    # nothing to do: no tensors, or only empty ones (their pointers are never read)
    assert L.roi_mask_fwd_grouped(None, 0, 2, 4, 1.0, 1.0, 0, 0, None) == roi.ROI_OK
    empty = [fwd_desc(0, rows=0, W=None, logits=None, W_masked=None), fwd_desc(1, cols=0)]
    assert grouped(L, fn, empty) == roi.ROI_OK


def test_bwd_grouped_rejects_before_launch(L):
    ok = [bwd_desc(0), bwd_desc(1)]
    cases = [
        ([ok[0], bwd_desc(1, cols=10)], roi.ROI_E_INVAL, "tensor 1"),
        ([ok[0], bwd_desc(1, d=None)], roi.ROI_E_INVAL, "tensor 1"),
        ([bwd_desc(0, G=FAKE + 2), ok[1]], roi.ROI_E_INVAL, "tensor 0"),
        ([ok[0], bwd_desc(1, d=FAKE + 2 * GB)], roi.ROI_E_INVAL, "overlap"),  # logits of tensor 0
        ([bwd_desc(0, W=FAKE + 8 * GB + GB), ok[1]], roi.ROI_E_INVAL, None),  # shared input: fine,
    ]
    for descs, status, msg in cases[:-1]:
        assert grouped(L, "roi_mask_bwd_grouped", descs) == status
        assert msg in L.roi_last_error().decode()
    # inputs may be shared between tensors; the call still fails here, on the
    # unsupported pattern, before anything is launched
    assert grouped(L, "roi_mask_bwd_grouped", cases[-1][0], m=64, n=2) == roi.ROI_E_UNSUPPORTED
    assert L.roi_mask_bwd_grouped(None, 0, 2, 4, 1.0, 1.0, 0, 0, None) == roi.ROI_OK
    assert L.roi_mask_bwd_grouped(None, 3, 2, 4, 1.0, 1.0, 0, 0, None) == roi.ROI_E_INVAL


def adamw(L, opt, **kw):
    a = dict(G=FAKE, W=FAKE + GB, logits=FAKE + 2 * GB, ea=FAKE + 3 * GB, eas=FAKE + 4 * GB,
             d=None, rows=4, cols=8, n=2, m=4, tau=1.0, lam=1.0, off=0)
    a.update(kw)
    return L.roi_mask_bwd_adamw(a["G"], a["W"], a["logits"], a["ea"], a["eas"], a["d"],
                                a["rows"], a["cols"], a["n"], a["m"], a["tau"], a["lam"], 0, 0,
                                a["off"], None if opt is None else ctypes.addressof(opt), None)


@pytest.mark.parametrize("okw,kw,status", [
    (None, {}, roi.ROI_E_INVAL),                               # no parameters
    (dict(lr=-1e-3), {}, roi.ROI_E_INVAL),
    (dict(lr=math.nan), {}, roi.ROI_E_INVAL),
    (dict(lr=math.inf), {}, roi.ROI_E_INVAL),
    (dict(betas=(1.0, 0.95)), {}, roi.ROI_E_INVAL),
    (dict(betas=(0.9, -0.1)), {}, roi.ROI_E_INVAL),
    (dict(eps=0.0), {}, roi.ROI_E_INVAL),
    (dict(weight_decay=-0.05), {}, roi.ROI_E_INVAL),
    (dict(t=0), {}, roi.ROI_E_INVAL),
    ({}, dict(ea=None), roi.ROI_E_INVAL),
    ({}, dict(eas=None), roi.ROI_E_INVAL),
    ({}, dict(logits=None), roi.ROI_E_INVAL),
    ({}, dict(ea=FAKE + 3 * GB + 4), roi.ROI_E_INVAL),         # misaligned
    ({}, dict(ea=FAKE + 2 * GB + 16), roi.ROI_E_INVAL),        # moments overlap the logits
    ({}, dict(d=FAKE + 4 * GB), roi.ROI_E_INVAL),              # gradient over the second moment
    ({}, dict(W=FAKE + 2 * GB + 32), roi.ROI_E_INVAL),         # input inside the updated logits
    ({}, dict(cols=6), roi.ROI_E_INVAL),
    ({}, dict(m=64, n=2, cols=64), roi.ROI_E_UNSUPPORTED),
])
def test_bwd_adamw_rejects_before_launch(L, okw, kw, status):
    opt = None if okw is None else roi.adamw_params(**{"lr": 1e-3, **okw})
    assert adamw(L, opt, **kw) == status
    assert L.roi_last_error()


def test_bwd_adamw_grouped_rejects_before_launch(L):
    opt = roi.adamw_params(1e-3)
    bad = roi.adamw_params(1e-3, t=0)

    def desc(i, **kw):
        base = FAKE + i * 8 * GB
        a = dict(G=base, W=base + GB, logits=base + 2 * GB, ea=base + 3 * GB, eas=base + 4 * GB,
                 d=None, rows=4, cols=8, off=i * 32)
        a.update(kw)
        return roi.AdamWTensor(a["G"], a["W"], a["logits"], a["ea"], a["eas"], a["d"], a["rows"],
                               a["cols"], a["off"])

    def call(descs, o):
        arr = (roi.AdamWTensor * max(1, len(descs)))(*descs)
        return L.roi_mask_bwd_adamw_grouped(ctypes.addressof(arr), len(descs), 2, 4, 1.0, 1.0, 0,
                                            0, None if o is None else ctypes.addressof(o), None)

    assert call([desc(0), desc(1)], None) == roi.ROI_E_INVAL
    assert call([desc(0), desc(1)], bad) == roi.ROI_E_INVAL
    assert call([desc(0), desc(1, eas=None)], opt) == roi.ROI_E_INVAL
    assert "tensor 1" in L.roi_last_error().decode()
    assert call([desc(0), desc(1, ea=FAKE + 3 * GB)], opt) == roi.ROI_E_INVAL  # shared moment
    assert "overlap" in L.roi_last_error().decode()
    assert L.roi_mask_bwd_adamw_grouped(None, 0, 2, 4, 1.0, 1.0, 0, 0, ctypes.addressof(opt),
                                        None) == roi.ROI_OK
    assert L.roi_mask_bwd_adamw_grouped(None, -1, 2, 4, 1.0, 1.0, 0, 0, ctypes.addressof(opt),
                                        None) == roi.ROI_E_INVAL


def export(L, **kw):
    a = dict(logits=FAKE, W=FAKE + GB, rows=4, cols=8, n=2, m=4, Wm=FAKE + 2 * GB,
             vals=FAKE + 3 * GB, idx=FAKE + 4 * GB, meta=None)
    a.update(kw)
    return L.roi_mask_export(a["logits"], a["W"], a["rows"], a["cols"], a["n"], a["m"], a["Wm"],
                             a["vals"], a["idx"], a["meta"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(meta=FAKE + 5 * GB, n=4, m=8), roi.ROI_E_INVAL),   # metadata only for 2:4
    (dict(Wm=None, vals=None, idx=None), roi.ROI_E_INVAL),  # nothing requested
    (dict(logits=None), roi.ROI_E_INVAL),
    (dict(W=None), roi.ROI_E_INVAL),                        # W needed for weight outputs
    (dict(W=FAKE + GB + 2), roi.ROI_E_INVAL),
    (dict(vals=FAKE + GB + 8), roi.ROI_E_INVAL),            # overlaps W
    (dict(idx=FAKE + 3 * GB + 4 * 2), roi.ROI_E_INVAL),    # misaligned
    (dict(idx=FAKE + 3 * GB), roi.ROI_E_INVAL),             # same address as the values
    (dict(cols=6), roi.ROI_E_INVAL),
    (dict(m=12, n=2, cols=12), roi.ROI_E_UNSUPPORTED),
    (dict(n=0), roi.ROI_E_INVAL),
])
def test_export_rejects_before_launch(L, kw, status):
    assert export(L, **kw) == status
    assert L.roi_last_error()


def test_export_empty_is_a_no_op(L):
    assert export(L, rows=0, logits=None, W=None, Wm=None, vals=None, idx=FAKE) == roi.ROI_OK


def test_cat_candidates_and_rejections(L):
    import math as _m
    for m in (4, 8):
        for n in range(1, m + 1):
            assert L.roi_cat_num_candidates(n, m) == _m.comb(m, n)
    assert L.roi_cat_num_candidates(2, 16) == -1 and L.roi_cat_num_candidates(0, 4) == -1

    def fwd(**kw):
        a = dict(W=FAKE, al=FAKE + GB, rows=4, cols=8, n=2, m=4, tau=1.0, lam=1.0, off=0,
                 Wm=FAKE + 2 * GB, S=None, ch=None)
        a.update(kw)
        return L.roi_cat_mask_fwd(a["W"], a["al"], a["rows"], a["cols"], a["n"], a["m"],
                                  a["tau"], a["lam"], 0, 0, a["off"], a["Wm"], a["S"], a["ch"],
                                  None)

    def bwd(**kw):
        a = dict(G=FAKE, W=FAKE + GB, al=FAKE + 2 * GB, rows=4, cols=8, n=2, m=4, tau=1.0,
                 lam=1.0, off=0, d=FAKE + 3 * GB)
        a.update(kw)
        return L.roi_cat_mask_bwd(a["G"], a["W"], a["al"], a["rows"], a["cols"], a["n"], a["m"],
                                  a["tau"], a["lam"], 0, 0, a["off"], a["d"], None)

    for f, kw, st in [
        (fwd, dict(m=16, n=2, cols=16), roi.ROI_E_UNSUPPORTED),
        (fwd, dict(n=5), roi.ROI_E_INVAL), (fwd, dict(cols=6), roi.ROI_E_INVAL),
        (fwd, dict(tau=0.0), roi.ROI_E_INVAL), (fwd, dict(lam=math.nan), roi.ROI_E_INVAL),
        (fwd, dict(Wm=None), roi.ROI_E_INVAL), (fwd, dict(al=FAKE + GB + 8), roi.ROI_E_INVAL),
        (fwd, dict(Wm=FAKE + GB + 16), roi.ROI_E_INVAL),        # overlaps the logits
        (fwd, dict(off=2 ** 64 - 4), roi.ROI_E_INVAL),          # noise index overflow
        (bwd, dict(d=None), roi.ROI_E_INVAL), (bwd, dict(d=FAKE + 2 * GB + 16), roi.ROI_E_INVAL),
        (bwd, dict(m=32, n=2, cols=32), roi.ROI_E_UNSUPPORTED), (bwd, dict(rows=-1), roi.ROI_E_INVAL),
    ]:
        assert f(**kw) == st, kw
        assert L.roi_last_error()
    assert fwd(rows=0, W=None, al=None, Wm=None) == roi.ROI_OK


def test_empty_input_is_a_no_op(L):
    # nothing to do: returns OK without touching the (NULL) pointers or the device
    assert fwd(L, rows=0, W=None, logits=None, Wm=None) == roi.ROI_OK
    assert fwd(L, cols=0, W=None, logits=None, Wm=None) == roi.ROI_OK
    assert bwd(L, rows=0, G=None, W=None, logits=None, d=None) == roi.ROI_OK
    assert L.roi_gumbel_noise(0, 0, 0, 0, None, None, None) == roi.ROI_OK
    assert L.roi_gumbel_from_words(None, 0, None, None) == roi.ROI_OK
    assert L.roi_fast_noise_from_words(None, 0, None, None) == roi.ROI_OK


def test_noise_entry_checks(L):
    assert L.roi_gumbel_noise(0, 0, 2, 16, FAKE, None, None) == roi.ROI_E_INVAL
    assert L.roi_gumbel_noise(0, 0, 0, 16, None, None, None) == roi.ROI_E_INVAL
    assert L.roi_gumbel_noise(0, 0, 0, -1, FAKE, None, None) == roi.ROI_E_INVAL
    assert L.roi_gumbel_noise(0, 0, 0, 16, FAKE, FAKE + 32, None) == roi.ROI_E_INVAL
    assert L.roi_gumbel_from_words(FAKE, 8, FAKE + 16, None) == roi.ROI_E_INVAL
    assert L.roi_gumbel_from_words(FAKE + 4, 8, FAKE + 4096, None) == roi.ROI_E_INVAL
    assert L.roi_fast_noise_from_words(FAKE, 8, FAKE + 16, None) == roi.ROI_E_INVAL   # overlap
    assert L.roi_fast_noise_from_words(FAKE + 4, 8, FAKE + 4096, None) == roi.ROI_E_INVAL
    assert L.roi_fast_noise_from_words(FAKE, -1, FAKE + 4096, None) == roi.ROI_E_INVAL
    assert L.roi_fast_noise_from_words(None, 8, FAKE + 4096, None) == roi.ROI_E_INVAL


def test_anneal_matches_oracle(L):
    """§4.2.3 schedule: the library's host function against the oracle's."""
    import oracle
    for (a, b, T) in ((1.0, 0.1, 9), (1.0, 0.05, 1500), (1.0, 0.002, 1500), (0.5, 2.0, 10)):
        for t in (0, 1, 2, T // 2, T - 1, T, T + 1, 3 * T):
            ref = oracle.anneal(a, b, t, T)
            got = roi.anneal(a, b, t, T)
            assert got == pytest.approx(ref, rel=1e-6), (a, b, T, t)
    assert math.isnan(roi.anneal(0.0, 0.1, 1, 9))
    assert math.isnan(roi.anneal(1.0, 0.1, 1, 0))
    assert math.isnan(roi.anneal(1.0, 0.1, -1, 9))


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(roi, "_lib", None)
    monkeypatch.setattr(roi, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        roi.lib()
