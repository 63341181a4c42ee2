"""Seeded synthetic inputs for the K-VEC eviction step (shared by the oracle
side and the GPU side; holds none of the eviction arithmetic).

The generator itself is C (``synth.c``, built into ``_synth.so``) so that a
full Llama-3.1-8B-shaped cache (up to 17 GB of K and V) can be produced in
seconds and any slice can be regenerated bit-identically for the oracle.

Workload table: the five shapes the eviction step is measured on.  Method
hyper-parameters follow the paper's implementation details: delta = 3 heads,
lambda = 1.0 (Sec. 5.1), beta = 0.25 (ablation table, retention ratio), and an
extended window O' = 2 * O (the paper's 16 -> 32 ratio, Sec. 4.1 and 5.1).
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, replace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_synth.so")
_SRC = os.path.join(_HERE, "synth.c")


def build(force: bool = True) -> str:
    """Compile synth.c into _synth.so (gcc, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-ffp-contract=off", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Cfg(ctypes.Structure):
    _fields_ = [
        ("seed", ctypes.c_uint64),
        ("n_layers", ctypes.c_int32), ("batch", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("seq_len", ctypes.c_int32),
        ("window", ctypes.c_int32), ("window_ext", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("rope", ctypes.c_int32),
        ("rope_theta", ctypes.c_double),
        ("hh_count", ctypes.c_int32), ("hh_shared", ctypes.c_int32),
        ("hh_scale", ctypes.c_double),
        ("sink_count", ctypes.c_int32), ("sink_scale", ctypes.c_double),
        ("zipf_clusters", ctypes.c_int32), ("zipf_s", ctypes.c_double),
    ]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.POINTER(_Cfg)
        i = ctypes.c_int
        lib.synth_keys.argtypes = [P, i, i, i, i, i, i, ctypes.c_void_p]
        lib.synth_values.argtypes = [P, i, i, i, i, i, i, ctypes.c_void_p]
        lib.synth_queries.argtypes = [P, i, i, i, i, ctypes.c_void_p]
        lib.synth_hh_positions.argtypes = [P, i, i, i, ctypes.c_void_p, i]
        lib.synth_hh_positions.restype = ctypes.c_int
        _lib = lib
    return _lib


@dataclass(frozen=True)
class Workload:
    """Shape, input recipe and method hyper-parameters of one workload."""
    name: str
    n_layers: int
    n_kv_heads: int
    n_q_heads: int
    head_dim: int
    seq_len: int
    batch: int
    window: int            # O
    window_ext: int        # O'
    budget: int            # B per KV head, including the window
    pool_kernel: int
    dtype: str             # "bf16" or "f32"
    seed: int
    rope: bool = True
    rope_theta: float = 500000.0
    hh_count: int = 0
    hh_shared: int = 0
    hh_scale: float = 4.0
    sink_count: int = 0
    sink_scale: float = 6.0
    zipf_clusters: int = 0
    zipf_s: float = 1.1
    n_adjust_heads: int = 3   # delta
    lam: float = 1.0          # lambda
    beta: float = 0.25
    criterion: str = "std"    # head focus criterion of H_top: "std" or "entropy"

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def rows(self) -> int:
        """Number of generated query rows, O' clamped to T."""
        return min(self.window_ext, self.seq_len)

    @property
    def candidates(self) -> int:
        return max(self.seq_len - self.window, 0)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def _hh(frac: float, T: int) -> int:
    return int(round(frac * T))


# The measured workloads.  Heavy-hitter counts are fractions of the prefix
# length T: 2% (tiny, 4k), 1% (32k), 2% with an 80% shared core (16k x 8),
# 0.5% from a Zipf(1.1) over 256 clusters (128k).
WORKLOADS = {
    0: Workload("tiny-fp32", 2, 4, 8, 64, 1024, 1, 32, 64, 128, 7, "f32", 1000,
                rope=False, hh_count=_hh(0.02, 1024)),
    1: Workload("llama8b-4k", 32, 8, 32, 128, 4096, 1, 32, 64, 128, 7, "bf16", 1001,
                hh_count=_hh(0.02, 4096)),
    2: Workload("llama8b-32k", 32, 8, 32, 128, 32768, 1, 32, 64, 1024, 7, "bf16", 1002,
                hh_count=_hh(0.01, 32768), sink_count=64),
    3: Workload("llama8b-16k-b8", 32, 8, 32, 128, 16384, 8, 64, 128, 512, 5, "bf16", 1003,
                hh_count=_hh(0.02, 16384), hh_shared=int(0.8 * _hh(0.02, 16384))),
    4: Workload("llama8b-128k", 32, 8, 32, 128, 131072, 1, 32, 64, 2048, 7, "bf16", 1004,
                hh_count=_hh(0.005, 131072), zipf_clusters=256),
    # The paper's second model (Qwen2.5-7B-Instruct, Sec. 5.3): 28 layers, 4 KV
    # and 28 query heads (GQA group 7), d = 128, RoPE theta 1e6; the 32k recipe.
    5: Workload("qwen7b-32k", 28, 4, 28, 128, 32768, 1, 32, 64, 1024, 7, "bf16", 1005,
                rope_theta=1000000.0, hh_count=_hh(0.01, 32768), sink_count=64),
}


def workload(i: int) -> Workload:
    return WORKLOADS[i]


def _cfg(w: Workload) -> _Cfg:
    return _Cfg(seed=w.seed, n_layers=w.n_layers, batch=w.batch, n_kv_heads=w.n_kv_heads,
                n_q_heads=w.n_q_heads, head_dim=w.head_dim, seq_len=w.seq_len,
                window=w.window, window_ext=w.window_ext,
                dtype=0 if w.dtype == "bf16" else 1, rope=1 if w.rope else 0,
                rope_theta=w.rope_theta, hh_count=w.hh_count, hh_shared=w.hh_shared,
                hh_scale=w.hh_scale, sink_count=w.sink_count, sink_scale=w.sink_scale,
                zipf_clusters=w.zipf_clusters, zipf_s=w.zipf_s)


def _storage(w: Workload):
    return np.uint16 if w.dtype == "bf16" else np.float32


def _ptr(a: np.ndarray) -> int:
    assert a.flags.c_contiguous
    return a.ctypes.data


def keys(w: Workload, layer: int, b: int, h0: int = 0, h1: int | None = None,
         t0: int = 0, t1: int | None = None, out: np.ndarray | None = None) -> np.ndarray:
    """K rows [h1-h0][t1-t0][d] (bf16 as uint16 bit patterns, or fp32)."""
    h1 = w.n_kv_heads if h1 is None else h1
    t1 = w.seq_len if t1 is None else t1
    shape = (h1 - h0, t1 - t0, w.head_dim)
    if out is None:
        out = np.empty(shape, dtype=_storage(w))
    assert out.shape == shape and out.dtype == _storage(w)
    c = _cfg(w)
    _load().synth_keys(ctypes.byref(c), layer, b, h0, h1, t0, t1, _ptr(out))
    return out


def values(w: Workload, layer: int, b: int, h0: int = 0, h1: int | None = None,
           t0: int = 0, t1: int | None = None, out: np.ndarray | None = None) -> np.ndarray:
    h1 = w.n_kv_heads if h1 is None else h1
    t1 = w.seq_len if t1 is None else t1
    shape = (h1 - h0, t1 - t0, w.head_dim)
    if out is None:
        out = np.empty(shape, dtype=_storage(w))
    assert out.shape == shape and out.dtype == _storage(w)
    c = _cfg(w)
    _load().synth_values(ctypes.byref(c), layer, b, h0, h1, t0, t1, _ptr(out))
    return out


def queries(w: Workload, layer: int, b: int, j0: int = 0, j1: int | None = None,
            out: np.ndarray | None = None) -> np.ndarray:
    """Q window rows [j1-j0][O'][d] at positions T-O'..T-1."""
    j1 = w.n_q_heads if j1 is None else j1
    shape = (j1 - j0, w.rows, w.head_dim)
    if out is None:
        out = np.empty(shape, dtype=_storage(w))
    assert out.shape == shape and out.dtype == _storage(w)
    c = _cfg(w)
    _load().synth_queries(ctypes.byref(c), layer, b, j0, j1, _ptr(out))
    return out


def hh_positions(w: Workload, layer: int, b: int, h: int) -> np.ndarray:
    cap = max(w.hh_count, 1)
    out = np.empty(cap, dtype=np.int32)
    c = _cfg(w)
    n = _load().synth_hh_positions(ctypes.byref(c), layer, b, h, _ptr(out), cap)
    return out[:min(n, cap)].copy()


def to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact conversion of generator storage to float64."""
    if dtype == "bf16":
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)
