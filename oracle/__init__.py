"""Plain CPU oracle of the RoI N:M mask sampler (arxiv 2608.23048).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package.  It shares no code with the HIP library in
``paper_2608_23048_amd``; both follow the same written definitions (see
``roi_oracle.c`` for the per-step citations of the paper).

This module only marshals numpy arrays into the C oracle (``roi_oracle.c``),
which is built with plain ``gcc`` and IEEE semantics (no contraction, no fast
math) so that its fp32 keys are one well-defined value per input.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "roi_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

GCC_FLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
             "-fno-strict-aliasing", "-Wall", "-Wextra"]


def build(verbose: bool = False) -> str:
    """Compile ``liboracle.so`` with gcc (always recompiles)."""
    tmp = f"{_LIB_PATH}.tmp{os.getpid()}"
    cmd = ["gcc", *GCC_FLAGS, _SRC, "-o", tmp, "-lm", "-lpthread"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None

_u8p = ctypes.POINTER(ctypes.c_uint8)
_u16p = ctypes.POINTER(ctypes.c_uint16)
_u32p = ctypes.POINTER(ctypes.c_uint32)
_u64p = ctypes.POINTER(ctypes.c_uint64)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_i64 = ctypes.c_int64
_u64 = ctypes.c_uint64
_int = ctypes.c_int
_f32 = ctypes.c_float
_f64 = ctypes.c_double


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        L.oracle_philox4x32_10.argtypes = [_u32p, _u32p, _u32p]
        L.oracle_philox4x32_10.restype = None
        L.oracle_philox_word.argtypes = [_u64, _u64, _u64]
        L.oracle_philox_word.restype = ctypes.c_uint32
        L.oracle_uniform.argtypes = [ctypes.c_uint32]
        L.oracle_uniform.restype = _f32
        L.oracle_log.argtypes = [_f32]
        L.oracle_log.restype = _f32
        L.oracle_log_array.argtypes = [_f32p, _i64, _f32p]
        L.oracle_log_array.restype = None
        L.oracle_gumbel.argtypes = [_f32]
        L.oracle_gumbel.restype = _f32
        L.oracle_gumbel_from_words.argtypes = [_u32p, _i64, _f32p]
        L.oracle_gumbel_from_words.restype = None
        L.oracle_keys.argtypes = [_f32p, _i64, _f32, _u64, _u64, _u64, _f32p]
        L.oracle_keys.restype = None
        L.oracle_topn.argtypes = [_f32p, _int, _int, _u8p, _u8p]
        L.oracle_topn.restype = _int
        L.oracle_relax_fwd.argtypes = [_f64p, _int, _int, _f64, _f64p]
        L.oracle_relax_fwd.restype = _int
        L.oracle_relax_bwd.argtypes = [_f64p, _int, _int, _f64, _f64p, _f64p]
        L.oracle_relax_bwd.restype = _int
        L.roi_oracle_fwd.argtypes = [_u16p, _f32p, _i64, _int, _int, _f32, _f32, _u64, _u64, _u64,
                                     _u16p, _f64p, _u8p]
        L.roi_oracle_fwd.restype = _int
        L.roi_oracle_bwd.argtypes = [_u16p, _u16p, _f32p, _i64, _int, _int, _f32, _f32, _u64,
                                     _u64, _u64, _f64p]
        L.roi_oracle_bwd.restype = _int
        L.roi_oracle_fwd_groups.argtypes = [_u16p, _f32p, _i64, _u64p, _int, _int, _f32, _f32,
                                            _u64, _u64, _u16p, _f64p, _u8p]
        L.roi_oracle_fwd_groups.restype = _int
        L.roi_oracle_bwd_groups.argtypes = [_u16p, _u16p, _f32p, _i64, _u64p, _int, _int, _f32,
                                            _f32, _u64, _u64, _f64p]
        L.roi_oracle_bwd_groups.restype = _int
        L.roi_oracle_fwd_mt.argtypes = [_u16p, _f32p, _i64, _int, _int, _f32, _f32, _u64, _u64,
                                        _u64, _u16p, _f64p, _u8p, _int]
        L.roi_oracle_fwd_mt.restype = _int
        L.roi_oracle_bwd_mt.argtypes = [_u16p, _u16p, _f32p, _i64, _int, _int, _f32, _f32, _u64,
                                        _u64, _u64, _f64p, _int]
        L.roi_oracle_bwd_mt.restype = _int
        L.oracle_relax_bwd_groups.argtypes = [_f64p, _i64, _int, _int, _f64, _f64p, _f64p, _int]
        L.oracle_relax_bwd_groups.restype = _int
        L.oracle_anneal.argtypes = [_f64, _f64, _f64, _f64]
        L.oracle_anneal.restype = _f64
        L.oracle_adamw.argtypes = [_f64p, _i64, _f64, _f64, _f64, _f64, _f64, _i64, _f32p, _f32p,
                                   _f32p, _f64p, _f64p, _f64p]
        L.oracle_adamw.restype = _int
        L.oracle_export.argtypes = [_f32p, _u16p, _i64, _int, _int, _u16p, _u16p, _u8p,
                                    ctypes.POINTER(ctypes.c_uint32)]
        L.oracle_export.restype = _int
        L.oracle_cat_candidates.argtypes = [_int, _int, ctypes.POINTER(ctypes.c_uint32)]
        L.oracle_cat_candidates.restype = _int
        L.oracle_cat_fwd.argtypes = [_u16p, _f32p, _i64, _int, _int, _f32, _f32, _u64, _u64, _u64,
                                     _u16p, _f64p, _u8p]
        L.oracle_cat_fwd.restype = _int
        L.oracle_cat_bwd.argtypes = [_u16p, _u16p, _f32p, _i64, _int, _int, _f32, _f32, _u64,
                                     _u64, _u64, _f64p]
        L.oracle_cat_bwd.restype = _int
        _lib = L
    return _lib


def _ptr(a: np.ndarray | None, ctype):
    if a is None:
        return ctypes.cast(None, ctypes.POINTER(ctype))
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (rc={rc})")


# --------------------------------------------------------------------------- primitives
def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint32))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint32))
    out = np.zeros(4, dtype=np.uint32)
    lib().oracle_philox4x32_10(_ptr(c, ctypes.c_uint32), _ptr(k, ctypes.c_uint32),
                               _ptr(out, ctypes.c_uint32))
    return out


def philox_word(seed: int, step: int, elem: int) -> int:
    return int(lib().oracle_philox_word(seed, step, elem))


def uniform(word: int) -> float:
    return float(lib().oracle_uniform(word))


def log32(x: float) -> np.float32:
    return np.float32(lib().oracle_log(np.float32(x)))


def log32_array(x: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(a.shape, dtype=np.float32)
    lib().oracle_log_array(_ptr(a, ctypes.c_float), a.size, _ptr(out, ctypes.c_float))
    return out


def gumbel(u: float) -> np.float32:
    return np.float32(lib().oracle_gumbel(np.float32(u)))


def gumbel_from_words(words: np.ndarray) -> np.ndarray:
    w = np.ascontiguousarray(words, dtype=np.uint32)
    g = np.empty(w.shape, dtype=np.float32)
    lib().oracle_gumbel_from_words(_ptr(w, ctypes.c_uint32), w.size, _ptr(g, ctypes.c_float))
    return g


def keys(phi: np.ndarray, lam: float, seed: int, step: int, elem_offset: int) -> np.ndarray:
    p = np.ascontiguousarray(phi, dtype=np.float32)
    k = np.empty(p.shape, dtype=np.float32)
    lib().oracle_keys(_ptr(p, ctypes.c_float), p.size, lam, seed, step, elem_offset,
                      _ptr(k, ctypes.c_float))
    return k


def topn(kappa, n: int):
    k = np.ascontiguousarray(np.asarray(kappa, dtype=np.float32))
    m = k.size
    order = np.zeros(n, dtype=np.uint8)
    hard = np.zeros(m, dtype=np.uint8)
    _check(lib().oracle_topn(_ptr(k, ctypes.c_float), m, n, _ptr(order, ctypes.c_uint8),
                             _ptr(hard, ctypes.c_uint8)), "topn")
    return order, hard


def relax_fwd(kappa, n: int, tau: float) -> np.ndarray:
    k = np.ascontiguousarray(np.asarray(kappa, dtype=np.float64))
    S = np.zeros(k.size, dtype=np.float64)
    _check(lib().oracle_relax_fwd(_ptr(k, ctypes.c_double), k.size, n, tau,
                                  _ptr(S, ctypes.c_double)), "relax_fwd")
    return S


def relax_bwd(kappa, n: int, tau: float, sbar) -> np.ndarray:
    k = np.ascontiguousarray(np.asarray(kappa, dtype=np.float64))
    sb = np.ascontiguousarray(np.asarray(sbar, dtype=np.float64))
    d = np.zeros(k.size, dtype=np.float64)
    _check(lib().oracle_relax_bwd(_ptr(k, ctypes.c_double), k.size, n, tau,
                                  _ptr(sb, ctypes.c_double), _ptr(d, ctypes.c_double)),
           "relax_bwd")
    return d


def anneal(v_init: float, v_end: float, t: float, t_anneal: float) -> float:
    return float(lib().oracle_anneal(v_init, v_end, t, t_anneal))


def adamw(grad, phi, m, v, lr: float, beta1: float, beta2: float, eps: float,
          weight_decay: float, t: int):
    """One AdamW step (fp64) from the fp64 gradient and the fp32 logits and
    moments; returns (phi, m, v) in fp64."""
    g = np.ascontiguousarray(grad, dtype=np.float64).reshape(-1)
    p = np.ascontiguousarray(phi, dtype=np.float32).reshape(-1)
    mm = np.ascontiguousarray(m, dtype=np.float32).reshape(-1)
    vv = np.ascontiguousarray(v, dtype=np.float32).reshape(-1)
    assert g.size == p.size == mm.size == vv.size
    po, mo, vo = (np.empty(g.size, dtype=np.float64) for _ in range(3))
    _check(lib().oracle_adamw(_ptr(g, ctypes.c_double), g.size, lr, beta1, beta2, eps,
                              weight_decay, t, _ptr(p, ctypes.c_float), _ptr(mm, ctypes.c_float),
                              _ptr(vv, ctypes.c_float), _ptr(po, ctypes.c_double),
                              _ptr(mo, ctypes.c_double), _ptr(vo, ctypes.c_double)), "adamw")
    return po, mo, vo


def export(logits, W_bits, n: int, m: int, want_meta: bool = False):
    """Final mask: top-n of the logits per group.  Returns (W_masked bits,
    values bits [G, n], idx [G, n] ascending, meta uint32 [ceil(G/8)] or None)."""
    p = np.ascontiguousarray(logits, dtype=np.float32).reshape(-1)
    W = np.ascontiguousarray(W_bits, dtype=np.uint16).reshape(-1)
    assert p.size == W.size
    G = p.size // m
    Wm = np.empty(p.size, dtype=np.uint16)
    vals = np.empty((G, n), dtype=np.uint16)
    idx = np.empty((G, n), dtype=np.uint8)
    meta = np.empty((G + 7) // 8, dtype=np.uint32) if want_meta else None
    _check(lib().oracle_export(_ptr(p, ctypes.c_float), _ptr(W, ctypes.c_uint16), p.size, n, m,
                               _ptr(Wm, ctypes.c_uint16), _ptr(vals, ctypes.c_uint16),
                               _ptr(idx, ctypes.c_uint8), _ptr(meta, ctypes.c_uint32)), "export")
    return Wm, vals, idx, meta


def cat_candidates(n: int, m: int) -> np.ndarray:
    """The candidate masks of the categorical sampler (bitmasks, lexicographic)."""
    out = np.zeros(70, dtype=np.uint32)
    C = lib().oracle_cat_candidates(n, m, _ptr(out, ctypes.c_uint32))
    _check(0 if C > 0 else -1, "cat_candidates")
    return out[:C].copy()


def cat_fwd(W_bits, alpha, n: int, m: int, tau: float, lam: float, seed: int, step: int,
            group_offset: int = 0, want_soft: bool = True):
    """Categorical sampler forward: (W_masked bits, S fp64 or None, choice uint8 [G])."""
    C = cat_candidates(n, m).size
    W = np.ascontiguousarray(W_bits, dtype=np.uint16).reshape(-1)
    a = np.ascontiguousarray(alpha, dtype=np.float32).reshape(-1)
    G = W.size // m
    assert a.size == G * C
    Wm = np.empty(W.size, dtype=np.uint16)
    S = np.empty(W.size, dtype=np.float64) if want_soft else None
    ch = np.empty(G, dtype=np.uint8)
    _check(lib().oracle_cat_fwd(_ptr(W, ctypes.c_uint16), _ptr(a, ctypes.c_float), G, n, m, tau,
                                lam, seed, step, group_offset, _ptr(Wm, ctypes.c_uint16),
                                _ptr(S, ctypes.c_double), _ptr(ch, ctypes.c_uint8)), "cat_fwd")
    return Wm, S, ch


def cat_bwd(G_bits, W_bits, alpha, n: int, m: int, tau: float, lam: float, seed: int, step: int,
            group_offset: int = 0) -> np.ndarray:
    """Categorical sampler backward: dL/dalpha (fp64, [G * C])."""
    Gb = np.ascontiguousarray(G_bits, dtype=np.uint16).reshape(-1)
    W = np.ascontiguousarray(W_bits, dtype=np.uint16).reshape(-1)
    a = np.ascontiguousarray(alpha, dtype=np.float32).reshape(-1)
    d = np.empty(a.size, dtype=np.float64)
    _check(lib().oracle_cat_bwd(_ptr(Gb, ctypes.c_uint16), _ptr(W, ctypes.c_uint16),
                                _ptr(a, ctypes.c_float), W.size // m, n, m, tau, lam, seed, step,
                                group_offset, _ptr(d, ctypes.c_double)), "cat_bwd")
    return d


# --------------------------------------------------------------------------- whole arrays
# The CPU share of one GPU on the machines the suite runs on.
MAX_THREADS = 16


def host_threads() -> int:
    """Threads for the threaded oracle: the cores this process may run on,
    at most MAX_THREADS."""
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    return max(1, min(MAX_THREADS, n))


def mask_fwd(W_bits: np.ndarray, logits: np.ndarray, n: int, m: int, tau: float, lam: float,
             seed: int, step: int, elem_offset: int = 0, want_soft: bool = True,
             threads: int = 1):
    """Returns (W_masked bits uint16, soft mask float64 or None, sel_idx uint8 [G, n]).
    threads > 1 splits the groups over that many threads (same bits)."""
    W = np.ascontiguousarray(W_bits, dtype=np.uint16).reshape(-1)
    p = np.ascontiguousarray(logits, dtype=np.float32).reshape(-1)
    assert W.size == p.size
    numel = W.size
    Wm = np.empty(numel, dtype=np.uint16)
    S = np.empty(numel, dtype=np.float64) if want_soft else None
    idx = np.empty(numel // m * n, dtype=np.uint8)
    args = (_ptr(W, ctypes.c_uint16), _ptr(p, ctypes.c_float), numel, n, m, tau, lam, seed,
            step, elem_offset, _ptr(Wm, ctypes.c_uint16), _ptr(S, ctypes.c_double),
            _ptr(idx, ctypes.c_uint8))
    rc = lib().roi_oracle_fwd(*args) if threads <= 1 else lib().roi_oracle_fwd_mt(*args, threads)
    _check(rc, "fwd")
    return Wm, S, idx.reshape(-1, n)


def mask_bwd(G_bits: np.ndarray, W_bits: np.ndarray, logits: np.ndarray, n: int, m: int,
             tau: float, lam: float, seed: int, step: int, elem_offset: int = 0,
             threads: int = 1) -> np.ndarray:
    G = np.ascontiguousarray(G_bits, dtype=np.uint16).reshape(-1)
    W = np.ascontiguousarray(W_bits, dtype=np.uint16).reshape(-1)
    p = np.ascontiguousarray(logits, dtype=np.float32).reshape(-1)
    assert G.size == W.size == p.size
    d = np.empty(p.size, dtype=np.float64)
    args = (_ptr(G, ctypes.c_uint16), _ptr(W, ctypes.c_uint16), _ptr(p, ctypes.c_float), p.size,
            n, m, tau, lam, seed, step, elem_offset, _ptr(d, ctypes.c_double))
    rc = lib().roi_oracle_bwd(*args) if threads <= 1 else lib().roi_oracle_bwd_mt(*args, threads)
    _check(rc, "bwd")
    return d


def relax_bwd_groups(kappa, n: int, tau: float, sbar, threads: int = 1) -> np.ndarray:
    """The relaxation's backward on given keys: kappa, sbar [groups, m] (fp64);
    returns dL/dkappa [groups, m]."""
    k = np.ascontiguousarray(kappa, dtype=np.float64)
    sb = np.ascontiguousarray(sbar, dtype=np.float64)
    assert k.ndim == 2 and k.shape == sb.shape
    d = np.empty(k.shape, dtype=np.float64)
    _check(lib().oracle_relax_bwd_groups(_ptr(k, ctypes.c_double), k.shape[0], k.shape[1], n,
                                         tau, _ptr(sb, ctypes.c_double),
                                         _ptr(d, ctypes.c_double), max(1, threads)),
           "relax_bwd_groups")
    return d


def mask_fwd_groups(W_bits, logits, group_elem, n, m, tau, lam, seed, step, want_soft=True):
    """Forward on gathered groups; arrays are [ngroups, m], group_elem[q] is the
    global index of group q's first element."""
    W = np.ascontiguousarray(W_bits, dtype=np.uint16).reshape(-1)
    p = np.ascontiguousarray(logits, dtype=np.float32).reshape(-1)
    ge = np.ascontiguousarray(group_elem, dtype=np.uint64).reshape(-1)
    ng = ge.size
    assert W.size == p.size == ng * m
    Wm = np.empty(W.size, dtype=np.uint16)
    S = np.empty(W.size, dtype=np.float64) if want_soft else None
    idx = np.empty(ng * n, dtype=np.uint8)
    _check(lib().roi_oracle_fwd_groups(_ptr(W, ctypes.c_uint16), _ptr(p, ctypes.c_float), ng,
                                       _ptr(ge, ctypes.c_uint64), n, m, tau, lam, seed, step,
                                       _ptr(Wm, ctypes.c_uint16), _ptr(S, ctypes.c_double),
                                       _ptr(idx, ctypes.c_uint8)), "fwd_groups")
    return Wm.reshape(ng, m), (S.reshape(ng, m) if S is not None else None), idx.reshape(ng, n)


def mask_bwd_groups(G_bits, W_bits, logits, group_elem, n, m, tau, lam, seed, step):
    G = np.ascontiguousarray(G_bits, dtype=np.uint16).reshape(-1)
    W = np.ascontiguousarray(W_bits, dtype=np.uint16).reshape(-1)
    p = np.ascontiguousarray(logits, dtype=np.float32).reshape(-1)
    ge = np.ascontiguousarray(group_elem, dtype=np.uint64).reshape(-1)
    ng = ge.size
    assert G.size == W.size == p.size == ng * m
    d = np.empty(p.size, dtype=np.float64)
    _check(lib().roi_oracle_bwd_groups(_ptr(G, ctypes.c_uint16), _ptr(W, ctypes.c_uint16),
                                       _ptr(p, ctypes.c_float), ng, _ptr(ge, ctypes.c_uint64), n,
                                       m, tau, lam, seed, step, _ptr(d, ctypes.c_double)),
           "bwd_groups")
    return d.reshape(ng, m)
