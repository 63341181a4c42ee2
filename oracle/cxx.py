"""The C++ oracle (oracle/kvec_oracle.cpp) with the signatures of kvec_oracle.py.

TEST INFRASTRUCTURE ONLY, like kvec_oracle.py: imported by tests/, by the
smoke check and by the benchmark's CPU-baseline leg, never by the product
path.  The arithmetic is all in the C++ file; this module converts numpy
arrays and returns the same structures as kvec_oracle.py, so that one set of
checks pins both oracles and each is checked against the other.  The window
scores and row normalisers run on `threads` host threads (all CPUs this
process may use, by default).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .kvec_oracle import LayerResult

_DIR = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_DIR, "kvec_oracle.cpp")
_LIB_PATH = os.path.join(_DIR, "libkvec_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile kvec_oracle.cpp into libkvec_oracle.so (g++, no FMA contraction)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-pthread",
                               "-ffp-contract=off", _SRC, "-o", tmp])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        P, I, F, D = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_double
        lib.ko_window_scores.argtypes = [P, P, I, I, I, I, I, I, I, P, P, P, I]
        lib.ko_window_lse.argtypes = [P, P, I, I, I, I, I, P, I]
        lib.ko_maxpool.argtypes = [P, I, I, I, P]
        lib.ko_head_sigma.argtypes = [P, I, I, P]
        lib.ko_head_entropy.argtypes = [P, I, I, P]
        lib.ko_adjusted_heads.argtypes = [P, I, I, P]
        lib.ko_adjusted_heads.restype = I
        lib.ko_rank_first.argtypes = [P, I, I, P]
        lib.ko_preserve_count.argtypes = [I, I, F]
        lib.ko_preserve_count.restype = I
        lib.ko_adjusted_priority.argtypes = [P, P, P, I, F, P, I, I, P]
        lib.ko_select_layer.argtypes = [P, P, P, P, I, I, I, I, I, I, I, I, F, F, I,
                                        P, P, P, P, P, P, P]
        lib.ko_select_layer.restype = I
        lib.ko_counts_from_bits.argtypes = [P, I, I, P]
        lib.ko_coverage_count.argtypes = [P, I, I]
        lib.ko_coverage_count.restype = ctypes.c_int64
        lib.ko_gather_rows.argtypes = [P, P, I, I, I, I, P]
        lib.ko_decode_attention.argtypes = [P, P, P, P, I, I, I, I, P]
        _lib = lib
    return _lib


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


# S1 ------------------------------------------------------------------------

def window_scores(q_win, k, window: int, full: bool = False, threads: int | None = None):
    q = _c(q_win, np.float64)
    kk = _c(k, np.float64)
    hq, wn, d = q.shape
    hkv, T, _ = kk.shape
    n = T if full else T - window
    p = np.empty((hkv, n))
    pe = np.empty((hkv, n))
    imp = np.empty(n)
    _load().ko_window_scores(_p(q), _p(kk), hq, hkv, wn, T, d, window, int(full), _p(p), _p(pe),
                             _p(imp), threads or default_threads())
    return p, pe, imp


def window_lse(q_win, k, threads: int | None = None):
    q = _c(q_win, np.float64)
    kk = _c(k, np.float64)
    hq, wn, d = q.shape
    hkv, T, _ = kk.shape
    out = np.empty((hq, wn))
    _load().ko_window_lse(_p(q), _p(kk), hq, hkv, wn, T, d, _p(out), threads or default_threads())
    return out


def to_f32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def score_layer(q_win, k, window: int, threads: int | None = None):
    p, pe, imp = window_scores(q_win, k, window, threads=threads)
    return to_f32(p), to_f32(pe), to_f32(imp)


# S2 .. S6 ------------------------------------------------------------------

def maxpool1d(x, kernel: int):
    a = _c(x, np.float32)
    shp = a.shape
    a2 = a.reshape(-1, shp[-1])
    out = np.empty_like(a2)
    _load().ko_maxpool(_p(a2), a2.shape[0], a2.shape[1], int(kernel), _p(out))
    return out.reshape(shp)


def head_sigma(p):
    a = _c(p, np.float32)
    out = np.empty(a.shape[0])
    _load().ko_head_sigma(_p(a), a.shape[0], a.shape[1], _p(out))
    return out


def head_entropy(p):
    a = _c(p, np.float32)
    out = np.empty(a.shape[0])
    _load().ko_head_entropy(_p(a), a.shape[0], a.shape[1], _p(out))
    return out


def adjusted_heads(sigma, delta: int):
    key = _c(sigma, np.float64)
    out = np.empty(max(len(key), 1), dtype=np.int64)
    n = _load().ko_adjusted_heads(_p(key), len(key), int(delta), _p(out))
    return out[:n].copy()


def focus_heads(pooled, delta: int, criterion: str = "std"):
    if criterion == "std":
        return adjusted_heads(head_sigma(pooled), delta)
    if criterion == "entropy":
        return adjusted_heads(-head_entropy(pooled), delta)
    raise ValueError(criterion)


def rank_first(scores, k: int):
    a = _c(scores, np.float32)
    n = a.shape[0]
    k = max(0, min(int(k), n))
    out = np.empty(max(k, 1), dtype=np.int64)
    _load().ko_rank_first(_p(a), n, k, _p(out))
    return out[:k].copy()


def preserve_count(budget: int, window: int, beta: float) -> int:
    return int(_load().ko_preserve_count(int(budget), int(window), float(np.float32(beta))))


def adjusted_priority(p_sel, imp, n_t, layer: int, lam: float, keep):
    ps = _c(p_sel, np.float32)
    H, n = ps.shape
    out = np.empty_like(ps)
    _load().ko_adjusted_priority(_p(ps), _p(_c(imp, np.float32)), _p(_c(n_t, np.int64)), int(layer),
                                 float(np.float32(lam)), _p(_c(keep, np.uint8)), H, n, _p(out))
    return out


def select_layer(p_raw, p_ext_raw, imp, n_t, layer: int, *, T: int, window: int, window_ext: int,
                 budget: int, pool_kernel: int, delta: int, lam: float, beta: float,
                 criterion: str = "std") -> LayerResult:
    pr = _c(p_raw, np.float32)
    H = pr.shape[0]
    Tc = T - window
    ntc = max(Tc, 0)
    nt = _c(np.asarray(n_t)[:ntc], np.int64)
    idx = np.empty((H, budget), dtype=np.int32)
    htop = np.empty(max(H, 1), dtype=np.int64)
    sigma = np.empty(H)
    keep = np.empty((H, ntc), dtype=np.uint8)
    p_sel = np.empty((H, ntc), dtype=np.float32)
    p_adj = np.empty((H, ntc), dtype=np.float32)
    bits = np.empty(T, dtype=np.uint8)
    nh = _load().ko_select_layer(
        _p(pr), _p(_c(p_ext_raw, np.float32)), _p(_c(imp, np.float32)), _p(nt), int(layer), H, T,
        window, window_ext, budget, pool_kernel, delta, float(np.float32(lam)),
        float(np.float32(beta)), int(criterion == "entropy"), _p(idx), _p(htop), _p(sigma),
        _p(keep), _p(p_sel), _p(p_adj), _p(bits))
    return LayerResult(idx, htop[:nh].copy(), sigma, keep.astype(bool), p_sel, p_adj,
                       bits.astype(bool))


def evict_layer_from_scores(p_raw, p_ext_raw, imp, n_t, layer, w) -> LayerResult:
    return select_layer(p_raw, p_ext_raw, imp, n_t, layer, T=w.seq_len, window=w.window,
                        window_ext=w.window_ext, budget=w.budget, pool_kernel=w.pool_kernel,
                        delta=w.n_adjust_heads, lam=w.lam, beta=w.beta,
                        criterion=getattr(w, "criterion", "std"))


# S7, S8, decode --------------------------------------------------------------

def counts_from_bits(layer_bits_list):
    if len(layer_bits_list) == 0:
        return None
    b = _c(np.stack([np.asarray(x, dtype=bool) for x in layer_bits_list]), np.uint8)
    out = np.empty(b.shape[1], dtype=np.int64)
    _load().ko_counts_from_bits(_p(b), b.shape[0], b.shape[1], _p(out))
    return out


def layer_bits(idx, T: int):
    # the kept-token set of a layer, as ko_select_layer builds it
    bits = np.zeros(T, dtype=bool)
    v = np.asarray(idx)
    bits[v[v >= 0]] = True
    return bits


def coverage_count(layer_bits_list) -> int:
    b = _c(np.stack([np.asarray(x, dtype=bool) for x in layer_bits_list]), np.uint8)
    return int(_load().ko_coverage_count(_p(b), b.shape[0], b.shape[1]))


def gather_rows(x, idx):
    a = np.ascontiguousarray(x)
    ii = _c(idx, np.int32)
    H, B = ii.shape
    T = a.shape[1]
    row_bytes = int(np.prod(a.shape[2:], dtype=np.int64)) * a.itemsize
    out = np.empty((H, B) + a.shape[2:], dtype=a.dtype)
    _load().ko_gather_rows(_p(a), _p(ii), H, T, B, row_bytes, _p(out))
    return out


def decode_attention(q, k, v, valid=None):
    qq = _c(q, np.float64)
    kk = _c(k, np.float64)
    vv = _c(v, np.float64)
    hq, d = qq.shape
    hkv, n, _ = kk.shape
    out = np.empty((hq, d))
    va = None if valid is None else _c(valid, np.uint8)
    _load().ko_decode_attention(_p(qq), _p(kk), _p(vv), None if va is None else _p(va), hq, hkv, n, d,
                                _p(out))
    return out


__all__ = [
    "build", "window_scores", "window_lse", "to_f32", "score_layer", "maxpool1d", "head_sigma",
    "head_entropy", "adjusted_heads", "focus_heads", "rank_first", "preserve_count",
    "adjusted_priority", "select_layer", "evict_layer_from_scores", "counts_from_bits",
    "layer_bits", "coverage_count", "gather_rows", "decode_attention",
]
