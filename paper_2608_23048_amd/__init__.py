"""MI355X (gfx950) RoI differentiable N:M mask sampler.

Thin ctypes binding of ``libroi.so`` (declared in ``include/roi.h``): argument
marshalling only.  Every step of the sampler runs in the HIP kernels; torch is
used for device memory and the current stream.  If the library has not been
built, every call raises -- there is no other implementation behind it.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libroi.so")

ROI_OK = 0
ROI_E_INVAL = -1
ROI_E_UNSUPPORTED = -2
ROI_E_HIP = -3

SUPPORTED_M = (4, 8, 16, 32)


class RoiError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{detail} (status {status})")
        self.status = status


_lib = None


class FwdTensor(ctypes.Structure):
    """roi_fwd_tensor (include/roi.h)."""
    _fields_ = [("W", ctypes.c_void_p), ("logits", ctypes.c_void_p),
                ("W_masked", ctypes.c_void_p), ("soft_mask", ctypes.c_void_p),
                ("sel_idx", ctypes.c_void_p), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("elem_offset", ctypes.c_uint64)]


class AdamWParams(ctypes.Structure):
    """roi_adamw_params (include/roi.h)."""
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float), ("t", ctypes.c_int64)]


class AdamWTensor(ctypes.Structure):
    """roi_adamw_tensor (include/roi.h)."""
    _fields_ = [("grad_W_masked", ctypes.c_void_p), ("W", ctypes.c_void_p),
                ("logits", ctypes.c_void_p), ("exp_avg", ctypes.c_void_p),
                ("exp_avg_sq", ctypes.c_void_p), ("grad_logits", ctypes.c_void_p),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("elem_offset", ctypes.c_uint64)]


class BwdTensor(ctypes.Structure):
    """roi_bwd_tensor (include/roi.h)."""
    _fields_ = [("grad_W_masked", ctypes.c_void_p), ("W", ctypes.c_void_p),
                ("logits", ctypes.c_void_p), ("grad_logits", ctypes.c_void_p),
                ("rows", ctypes.c_int64), ("cols", ctypes.c_int64),
                ("elem_offset", ctypes.c_uint64)]

_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_u64 = ctypes.c_uint64
_int = ctypes.c_int
_f32 = ctypes.c_float


def lib() -> ctypes.CDLL:
    """The loaded libroi.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2608_23048_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.roi_mask_fwd.argtypes = [_vp, _vp, _i64, _i64, _int, _int, _f32, _f32, _u64, _u64, _u64,
                                   _vp, _vp, _vp, _vp]
        L.roi_mask_fwd.restype = _int
        L.roi_mask_fwd_soft.argtypes = L.roi_mask_fwd.argtypes
        L.roi_mask_fwd_soft.restype = _int
        L.roi_mask_bwd.argtypes = [_vp, _vp, _vp, _i64, _i64, _int, _int, _f32, _f32, _u64, _u64,
                                   _u64, _vp, _vp]
        L.roi_mask_bwd.restype = _int
        grouped = [_vp, _int, _int, _int, _f32, _f32, _u64, _u64, _vp]
        for name in ("roi_mask_fwd_grouped", "roi_mask_fwd_soft_grouped", "roi_mask_bwd_grouped"):
            getattr(L, name).argtypes = grouped
            getattr(L, name).restype = _int
        L.roi_mask_bwd_adamw.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _int, _int,
                                         _f32, _f32, _u64, _u64, _u64, _vp, _vp]
        L.roi_mask_bwd_adamw.restype = _int
        L.roi_mask_bwd_adamw_grouped.argtypes = [_vp, _int, _int, _int, _f32, _f32, _u64, _u64,
                                                 _vp, _vp]
        L.roi_mask_bwd_adamw_grouped.restype = _int
        L.roi_mask_export.argtypes = [_vp, _vp, _i64, _i64, _int, _int, _vp, _vp, _vp, _vp, _vp]
        L.roi_mask_export.restype = _int
        L.roi_cat_num_candidates.argtypes = [_int, _int]
        L.roi_cat_num_candidates.restype = _int
        L.roi_cat_mask_fwd.argtypes = [_vp, _vp, _i64, _i64, _int, _int, _f32, _f32, _u64, _u64,
                                       _u64, _vp, _vp, _vp, _vp]
        L.roi_cat_mask_fwd.restype = _int
        L.roi_cat_mask_bwd.argtypes = [_vp, _vp, _vp, _i64, _i64, _int, _int, _f32, _f32, _u64,
                                       _u64, _u64, _vp, _vp]
        L.roi_cat_mask_bwd.restype = _int
        L.roi_gumbel_noise.argtypes = [_u64, _u64, _u64, _i64, _vp, _vp, _vp]
        L.roi_gumbel_noise.restype = _int
        L.roi_gumbel_from_words.argtypes = [_vp, _i64, _vp, _vp]
        L.roi_gumbel_from_words.restype = _int
        L.roi_fast_noise_from_words.argtypes = [_vp, _i64, _vp, _vp]
        L.roi_fast_noise_from_words.restype = _int
        L.roi_stream_copy.argtypes = [_vp, _vp, _i64, _vp]
        L.roi_stream_copy.restype = _int
        L.roi_anneal.argtypes = [_f32, _f32, _i64, _i64]
        L.roi_anneal.restype = _f32
        L.roi_status_string.argtypes = [_int]
        L.roi_status_string.restype = ctypes.c_char_p
        L.roi_last_error.argtypes = []
        L.roi_last_error.restype = ctypes.c_char_p
        L.roi_abi_version.argtypes = []
        L.roi_abi_version.restype = _int
        _lib = L
    return _lib


def _raise_on(status: int):
    if status != ROI_OK:
        raise RoiError(status, lib().roi_last_error().decode() or
                       lib().roi_status_string(status).decode())


def _stream(t) -> int:
    import torch
    return torch.cuda.current_stream(t.device).cuda_stream


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _shape2d(t) -> tuple[int, int]:
    if t.dim() == 2:
        return int(t.shape[0]), int(t.shape[1])
    return 1, int(t.numel())


def _check_tensor(t, dtype, name, like=None):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if like is not None and t.shape != like.shape:
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(like.shape)}")


# --------------------------------------------------------------------------- tensor API
def mask_fwd(W, logits, n: int, m: int, tau: float = 1.0, lam: float = 1.0, seed: int = 0,
             step: int = 0, elem_offset: int = 0, want_soft: bool = False, want_idx: bool = True,
             out: dict | None = None, soft_forward: bool = False):
    """Forward sample.  W: bf16 [rows, cols] (or 1-D), logits: fp32 same shape.

    Returns (W_masked bf16, soft_mask fp32 or None, sel_idx uint8 [groups, n] or
    None).  ``out`` may hold preallocated "W_masked", "soft_mask", "sel_idx".
    soft_forward=False: straight-through forward, W_masked = W (.) hard mask;
    soft_forward=True: pure soft forward, W_masked = bf16(W (.) S).
    """
    import torch
    _check_tensor(W, torch.bfloat16, "W")
    _check_tensor(logits, torch.float32, "logits", like=W)
    rows, cols = _shape2d(W)
    out = out or {}
    Wm = out.get("W_masked")
    if Wm is None:
        Wm = torch.empty_like(W)
    S = out.get("soft_mask") if want_soft else None
    if want_soft and S is None:
        S = torch.empty_like(logits)
    idx = out.get("sel_idx") if want_idx else None
    if want_idx and idx is None:
        idx = torch.empty((W.numel() // m if m > 0 else 0, n), dtype=torch.uint8, device=W.device)
    fn = lib().roi_mask_fwd_soft if soft_forward else lib().roi_mask_fwd
    st = fn(_ptr(W), _ptr(logits), rows, cols, n, m, tau, lam, seed, step, elem_offset, _ptr(Wm),
            _ptr(S), _ptr(idx), _stream(W))
    _raise_on(st)
    return Wm, S, idx


def mask_bwd(grad_W_masked, W, logits, n: int, m: int, tau: float = 1.0, lam: float = 1.0,
             seed: int = 0, step: int = 0, elem_offset: int = 0, out=None):
    """dL/dlogits (fp32, same shape as logits) from dL/dW_masked (bf16)."""
    import torch
    _check_tensor(grad_W_masked, torch.bfloat16, "grad_W_masked")
    _check_tensor(W, torch.bfloat16, "W", like=grad_W_masked)
    _check_tensor(logits, torch.float32, "logits", like=grad_W_masked)
    rows, cols = _shape2d(W)
    d = out if out is not None else torch.empty_like(logits)
    st = lib().roi_mask_bwd(_ptr(grad_W_masked), _ptr(W), _ptr(logits), rows, cols, n, m, tau, lam,
                            seed, step, elem_offset, _ptr(d), _stream(W))
    _raise_on(st)
    return d


def adamw_params(lr: float, betas=(0.9, 0.95), eps: float = 1e-8, weight_decay: float = 0.05,
                 t: int = 1) -> AdamWParams:
    """AdamW settings of one step (defaults: the appendix's betas and weight decay)."""
    return AdamWParams(lr, betas[0], betas[1], eps, weight_decay, t)


def mask_bwd_adamw(grad_W_masked, W, logits, exp_avg, exp_avg_sq, n: int, m: int,
                   tau: float = 1.0, lam: float = 1.0, seed: int = 0, step: int = 0,
                   elem_offset: int = 0, opt: AdamWParams | None = None, grad_out=None):
    """Backward with the AdamW step on the logits fused in: logits, exp_avg and
    exp_avg_sq (fp32, shaped like W) are updated in place; grad_out (fp32,
    optional) also receives dL/dlogits.  Returns grad_out."""
    import torch
    _check_tensor(grad_W_masked, torch.bfloat16, "grad_W_masked")
    _check_tensor(W, torch.bfloat16, "W", like=grad_W_masked)
    for t, name in ((logits, "logits"), (exp_avg, "exp_avg"), (exp_avg_sq, "exp_avg_sq")):
        _check_tensor(t, torch.float32, name, like=grad_W_masked)
    if grad_out is not None:
        _check_tensor(grad_out, torch.float32, "grad_out", like=grad_W_masked)
    if opt is None:
        raise ValueError("opt (AdamWParams) is required")
    rows, cols = _shape2d(W)
    st = lib().roi_mask_bwd_adamw(_ptr(grad_W_masked), _ptr(W), _ptr(logits), _ptr(exp_avg),
                                  _ptr(exp_avg_sq), _ptr(grad_out), rows, cols, n, m, tau, lam,
                                  seed, step, elem_offset, ctypes.addressof(opt), _stream(W))
    _raise_on(st)
    return grad_out


def mask_bwd_adamw_grouped(tensors, n: int, m: int, tau: float = 1.0, lam: float = 1.0,
                           seed: int = 0, step: int = 0, offsets=None,
                           opt: AdamWParams | None = None, grad_outs=None):
    """mask_bwd_adamw over a list of (grad_W_masked, W, logits, exp_avg,
    exp_avg_sq) in one call (in place); grad_outs: optional list of fp32
    tensors receiving dL/dlogits."""
    import torch
    if opt is None:
        raise ValueError("opt (AdamWParams) is required")
    descs = []
    offs = _offsets([W.numel() for _, W, *_ in tensors], offsets)
    for i, ((G, W, logits, ea, eas), off) in enumerate(zip(tensors, offs)):
        _check_tensor(G, torch.bfloat16, "grad_W_masked")
        _check_tensor(W, torch.bfloat16, "W", like=G)
        for t, name in ((logits, "logits"), (ea, "exp_avg"), (eas, "exp_avg_sq")):
            _check_tensor(t, torch.float32, name, like=G)
        d = grad_outs[i] if grad_outs is not None else None
        rows, cols = _shape2d(W)
        descs.append(AdamWTensor(_ptr(G), _ptr(W), _ptr(logits), _ptr(ea), _ptr(eas), _ptr(d),
                                 rows, cols, off))
    arr = (AdamWTensor * max(1, len(descs)))(*descs)
    stream = _stream(tensors[0][1]) if tensors else 0
    _raise_on(lib().roi_mask_bwd_adamw_grouped(ctypes.addressof(arr), len(descs), n, m, tau, lam,
                                               seed, step, ctypes.addressof(opt), stream))


def mask_export(logits, W, n: int, m: int, want_dense: bool = True, want_values: bool = True,
                want_idx: bool = True, want_meta: bool = False):
    """Final mask (top-n of the logits per group): returns (W_masked, values
    [G, n], idx [G, n] increasing, meta uint32 [ceil(G/8)] for 2:4), each
    None unless requested."""
    import torch
    _check_tensor(logits, torch.float32, "logits")
    if W is not None:
        _check_tensor(W, torch.bfloat16, "W", like=logits)
    rows, cols = _shape2d(logits)
    G = logits.numel() // m if m > 0 else 0
    dev = logits.device
    Wm = torch.empty_like(W) if want_dense else None
    vals = torch.empty((G, n), dtype=torch.bfloat16, device=dev) if want_values else None
    idx = torch.empty((G, n), dtype=torch.uint8, device=dev) if want_idx else None
    meta = torch.empty(((G + 7) // 8,), dtype=torch.int32, device=dev) if want_meta else None
    _raise_on(lib().roi_mask_export(_ptr(logits), _ptr(W), rows, cols, n, m, _ptr(Wm), _ptr(vals),
                                    _ptr(idx), _ptr(meta), _stream(logits)))
    return Wm, vals, idx, meta


def cat_num_candidates(n: int, m: int) -> int:
    """binom(m, n): logits per group of the categorical sampler (-1 if not built)."""
    return int(lib().roi_cat_num_candidates(n, m))


def _check_cat(W, cat_logits, n, m):
    import torch
    _check_tensor(W, torch.bfloat16, "W")
    _check_tensor(cat_logits, torch.float32, "cat_logits")
    C = cat_num_candidates(n, m)
    if C < 1:
        raise RoiError(ROI_E_UNSUPPORTED, f"no categorical sampler for {n}:{m}")
    if cat_logits.numel() != (W.numel() // m) * C:
        raise ValueError(f"cat_logits must hold {C} logits per group of {m} weights")
    return C


def cat_mask_fwd(W, cat_logits, n: int, m: int, tau: float = 1.0, lam: float = 1.0,
                 seed: int = 0, step: int = 0, group_offset: int = 0, want_soft: bool = False,
                 want_choice: bool = True, out: dict | None = None):
    """Categorical sampler forward (one logit per candidate mask, [G, C] fp32):
    returns (W_masked bf16, soft mask fp32 or None, chosen candidate uint8 [G]
    or None)."""
    import torch
    _check_cat(W, cat_logits, n, m)
    rows, cols = _shape2d(W)
    out = out or {}
    Wm = out.get("W_masked")
    if Wm is None:
        Wm = torch.empty_like(W)
    S = out.get("soft_mask") if want_soft else None
    if want_soft and S is None:
        S = torch.empty(W.shape, dtype=torch.float32, device=W.device)
    ch = out.get("choice") if want_choice else None
    if want_choice and ch is None:
        ch = torch.empty(W.numel() // m, dtype=torch.uint8, device=W.device)
    _raise_on(lib().roi_cat_mask_fwd(_ptr(W), _ptr(cat_logits), rows, cols, n, m, tau, lam, seed,
                                     step, group_offset, _ptr(Wm), _ptr(S), _ptr(ch),
                                     _stream(W)))
    return Wm, S, ch


def cat_mask_bwd(grad_W_masked, W, cat_logits, n: int, m: int, tau: float = 1.0,
                 lam: float = 1.0, seed: int = 0, step: int = 0, group_offset: int = 0, out=None):
    """Categorical sampler backward: dL/dcat_logits (fp32, shaped like cat_logits)."""
    import torch
    _check_cat(W, cat_logits, n, m)
    _check_tensor(grad_W_masked, torch.bfloat16, "grad_W_masked", like=W)
    rows, cols = _shape2d(W)
    d = out if out is not None else torch.empty_like(cat_logits)
    _raise_on(lib().roi_cat_mask_bwd(_ptr(grad_W_masked), _ptr(W), _ptr(cat_logits), rows, cols,
                                     n, m, tau, lam, seed, step, group_offset, _ptr(d),
                                     _stream(W)))
    return d


def _offsets(sizes, offsets):
    if offsets is not None:
        if len(offsets) != len(sizes):
            raise ValueError("one elem_offset per tensor")
        return [int(o) for o in offsets]
    out, acc = [], 0
    for k in sizes:
        out.append(acc)
        acc += k
    return out


def mask_fwd_grouped(tensors, n: int, m: int, tau: float = 1.0, lam: float = 1.0, seed: int = 0,
                     step: int = 0, offsets=None, want_soft: bool = False, want_idx: bool = True,
                     soft_forward: bool = False, outs=None):
    """mask_fwd over a list of (W, logits) pairs in one call.  The element
    offsets default to the running sum of the sizes (a stack in list order).
    Returns a list of (W_masked, soft_mask or None, sel_idx or None); `outs`
    may hold such a list, preallocated."""
    import torch
    given, outs, descs = outs, [], []
    offs = _offsets([W.numel() for W, _ in tensors], offsets)
    for i, ((W, logits), off) in enumerate(zip(tensors, offs)):
        _check_tensor(W, torch.bfloat16, "W")
        _check_tensor(logits, torch.float32, "logits", like=W)
        rows, cols = _shape2d(W)
        if given is not None:
            Wm, S, idx = given[i]
            S = S if want_soft else None
            idx = idx if want_idx else None
        else:
            Wm = torch.empty_like(W)
            S = torch.empty_like(logits) if want_soft else None
            idx = (torch.empty((W.numel() // m if m > 0 else 0, n), dtype=torch.uint8,
                               device=W.device) if want_idx else None)
        outs.append((Wm, S, idx))
        descs.append(FwdTensor(_ptr(W), _ptr(logits), _ptr(Wm), _ptr(S), _ptr(idx), rows, cols,
                               off))
    arr = (FwdTensor * max(1, len(descs)))(*descs)
    fn = lib().roi_mask_fwd_soft_grouped if soft_forward else lib().roi_mask_fwd_grouped
    stream = _stream(tensors[0][0]) if tensors else 0
    _raise_on(fn(ctypes.addressof(arr), len(descs), n, m, tau, lam, seed, step, stream))
    return outs


def mask_bwd_grouped(tensors, n: int, m: int, tau: float = 1.0, lam: float = 1.0, seed: int = 0,
                     step: int = 0, offsets=None, outs=None):
    """mask_bwd over a list of (grad_W_masked, W, logits) triples in one call;
    returns the list of grad_logits (`outs`: preallocated, optional)."""
    import torch
    given, outs, descs = outs, [], []
    offs = _offsets([W.numel() for _, W, _ in tensors], offsets)
    for i, ((G, W, logits), off) in enumerate(zip(tensors, offs)):
        _check_tensor(G, torch.bfloat16, "grad_W_masked")
        _check_tensor(W, torch.bfloat16, "W", like=G)
        _check_tensor(logits, torch.float32, "logits", like=G)
        rows, cols = _shape2d(W)
        d = given[i] if given is not None else torch.empty_like(logits)
        _check_tensor(d, torch.float32, "grad_logits", like=logits)
        outs.append(d)
        descs.append(BwdTensor(_ptr(G), _ptr(W), _ptr(logits), _ptr(d), rows, cols, off))
    arr = (BwdTensor * max(1, len(descs)))(*descs)
    stream = _stream(tensors[0][1]) if tensors else 0
    _raise_on(lib().roi_mask_bwd_grouped(ctypes.addressof(arr), len(descs), n, m, tau, lam, seed,
                                         step, stream))
    return outs


def gumbel_noise(count: int, seed: int = 0, step: int = 0, elem_offset: int = 0, device="cuda",
                 want_words: bool = True, want_gumbel: bool = True):
    """Raw Philox words (as int32 bit patterns) and Gumbel noise of `count` elements."""
    import torch
    words = torch.empty(count, dtype=torch.int32, device=device) if want_words else None
    g = torch.empty(count, dtype=torch.float32, device=device) if want_gumbel else None
    ref = words if words is not None else g
    st = lib().roi_gumbel_noise(seed, step, elem_offset, count, _ptr(words), _ptr(g), _stream(ref))
    _raise_on(st)
    return words, g


def gumbel_from_words(words):
    """g = -L(-L(u(x))) for int32 tensors holding 32-bit words."""
    import torch
    _check_tensor(words, torch.int32, "words")
    g = torch.empty(words.shape, dtype=torch.float32, device=words.device)
    _raise_on(lib().roi_gumbel_from_words(_ptr(words), words.numel(), _ptr(g), _stream(words)))
    return g


def stream_copy(src, dst):
    """Plain streaming copy of src into dst (device tensors of the same byte
    size, a multiple of 16): the benchmark's data-movement reference."""
    if src.numel() * src.element_size() != dst.numel() * dst.element_size():
        raise ValueError("src and dst differ in size")
    _raise_on(lib().roi_stream_copy(_ptr(src), _ptr(dst), src.numel() * src.element_size(),
                                    _stream(src)))
    return dst


def fast_noise_from_words(words):
    """K = -log2(-log2 u(x)) from the hardware logarithm, for int32 word tensors."""
    import torch
    _check_tensor(words, torch.int32, "words")
    out = torch.empty(words.shape, dtype=torch.float32, device=words.device)
    _raise_on(lib().roi_fast_noise_from_words(_ptr(words), words.numel(), _ptr(out),
                                              _stream(words)))
    return out


def anneal(v_init: float, v_end: float, t: int, t_anneal: int) -> float:
    """§4.2.3 exponential annealing of a temperature (host-side)."""
    return float(lib().roi_anneal(v_init, v_end, t, t_anneal))
