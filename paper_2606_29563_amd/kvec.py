"""Thin Python binding of libkvec (argument marshalling only).

Every computation runs in the HIP library; this module converts torch tensors
to pointers, strides and the current HIP stream.  There is no CPU fallback: if
libkvec.so is missing or fails to load, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkvec.so")

KVEC_OK, KVEC_ERR_INVALID, KVEC_ERR_UNSUPPORTED, KVEC_ERR_WORKSPACE, KVEC_ERR_DEVICE = range(5)
KVEC_BF16, KVEC_F32 = 0, 1
KVEC_HEADS_STD, KVEC_HEADS_ENTROPY = 0, 1


class KvecError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} ({status})")


class kvec_config(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("n_layers", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("seq_len", ctypes.c_int32),
        ("window", ctypes.c_int32), ("window_ext", ctypes.c_int32),
        ("budget", ctypes.c_int32), ("pool_kernel", ctypes.c_int32),
        ("n_adjust_heads", ctypes.c_int32),
        ("lambda_", ctypes.c_float), ("beta", ctypes.c_float),
        ("dtype", ctypes.c_int32), ("head_criterion", ctypes.c_int32),
    ]


@dataclass
class Config:
    """Python view of kvec_config."""
    batch: int
    n_layers: int
    n_kv_heads: int
    n_q_heads: int
    head_dim: int
    seq_len: int
    window: int
    window_ext: int
    budget: int
    pool_kernel: int = 7
    n_adjust_heads: int = 3
    lam: float = 1.0
    beta: float = 0.25
    dtype: int = KVEC_BF16
    head_criterion: int = KVEC_HEADS_STD

    def c(self) -> kvec_config:
        return kvec_config(self.batch, self.n_layers, self.n_kv_heads, self.n_q_heads,
                           self.head_dim, self.seq_len, self.window, self.window_ext,
                           self.budget, self.pool_kernel, self.n_adjust_heads, self.lam,
                           self.beta, self.dtype, self.head_criterion)

    @classmethod
    def from_workload(cls, w, **over) -> "Config":
        kw = dict(batch=w.batch, n_layers=w.n_layers, n_kv_heads=w.n_kv_heads,
                  n_q_heads=w.n_q_heads, head_dim=w.head_dim, seq_len=w.seq_len,
                  window=w.window, window_ext=w.window_ext, budget=w.budget,
                  pool_kernel=w.pool_kernel, n_adjust_heads=w.n_adjust_heads, lam=w.lam,
                  beta=w.beta, dtype=KVEC_BF16 if w.dtype == "bf16" else KVEC_F32,
                  head_criterion=KVEC_HEADS_ENTROPY if getattr(w, "criterion", "std") == "entropy"
                  else KVEC_HEADS_STD)
        kw.update(over)
        return cls(**kw)

    @property
    def candidates(self) -> int:
        return self.seq_len - self.window

    @property
    def words(self) -> int:
        return (self.seq_len + 63) // 64


_lib = None

EXPORTS = ["kvec_workspace_size", "kvec_score", "kvec_score_lse", "kvec_select_cover",
           "kvec_compact", "kvec_evict_layer", "kvec_evict_model", "kvec_evict_model_lse",
           "kvec_evict_layer_lse", "kvec_evict_model_scores", "kvec_evict_model_steps",
           "kvec_evict_model_lse_steps",
           "kvec_profile_points", "kvec_profile_points_lse", "kvec_coverage",
           "kvec_decode_workspace_size", "kvec_decode_attention", "kvec_decode_attention_noalloc",
           "kvec_status_string"]


def load() -> ctypes.CDLL:
    """Load libkvec.so (building it first only if no build exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        from . import build as _build
        _build.build()
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER(kvec_config)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    I64x = ctypes.POINTER(ctypes.c_int64)
    lib.kvec_workspace_size.argtypes = [P, ctypes.POINTER(sz)]
    lib.kvec_score.argtypes = [P, vp, I64x, vp, I64x, vp, vp, vp, vp, sz, vp]
    lib.kvec_score_lse.argtypes = [P, vp, I64x, vp, I64x, vp, I64x, vp, vp, vp, vp, sz, vp]
    lib.kvec_select_cover.argtypes = [P, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.kvec_compact.argtypes = [P, vp, I64x, vp, I64x, vp, vp, vp, vp]
    lib.kvec_evict_layer.argtypes = [P, i32, vp, I64x, vp, I64x, vp, I64x, vp, vp, vp, vp, vp, sz, vp]
    lib.kvec_evict_model.argtypes = [P, vp, I64x, vp, I64x, vp, I64x, vp, vp, vp, vp, vp, sz, vp,
                                     ctypes.POINTER(vp)]
    lib.kvec_evict_layer_lse.argtypes = [P, i32, vp, I64x, vp, I64x, vp, I64x, vp, I64x, vp, vp,
                                         vp, vp, vp, sz, vp]
    lib.kvec_evict_model_lse.argtypes = [P, vp, I64x, vp, I64x, vp, I64x, vp, I64x, vp, vp, vp, vp,
                                         vp, sz, vp, ctypes.POINTER(vp)]
    lib.kvec_evict_model_scores.argtypes = [P, vp, I64x, vp, I64x, vp, I64x, vp, vp, vp, vp, vp,
                                            vp, vp, vp, vp, sz, vp]
    lib.kvec_evict_model_steps.argtypes = [P, i32, vp, I64x, vp, I64x, vp, I64x, vp, vp, vp, vp, vp,
                                           sz, vp]
    lib.kvec_evict_model_lse_steps.argtypes = [P, i32, vp, I64x, vp, I64x, vp, I64x, vp, I64x, vp, vp,
                                               vp, vp, vp, sz, vp]
    lib.kvec_decode_attention_noalloc.argtypes = [P, vp, I64x, vp, vp, I64x, i32, vp, vp, vp]
    lib.kvec_coverage.argtypes = [P, vp, i32, vp, vp]
    lib.kvec_decode_workspace_size.argtypes = [P, i32, ctypes.POINTER(sz)]
    lib.kvec_decode_attention.argtypes = [P, vp, I64x, vp, vp, I64x, i32, vp, vp, vp, sz, vp]
    lib.kvec_profile_points.argtypes = [P]
    lib.kvec_profile_points_lse.argtypes = [P]
    lib.kvec_status_string.argtypes = [ctypes.c_int]
    lib.kvec_status_string.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name not in ("kvec_status_string", "kvec_profile_points", "kvec_profile_points_lse"):
            getattr(lib, name).restype = ctypes.c_int
    lib.kvec_profile_points.restype = ctypes.c_int32
    lib.kvec_profile_points_lse.restype = ctypes.c_int32
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().kvec_status_string(status).decode()


def _check(status: int, what: str) -> None:
    if status != KVEC_OK:
        raise KvecError(status, what)


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _strides(t, n: int):
    """Element strides of the leading n dims of a tensor whose last dim is contiguous."""
    if t is None:
        return None
    assert t.stride(-1) == 1, "the head dimension must be contiguous"
    st = list(t.stride())[:n]
    return (ctypes.c_int64 * n)(*st)


def _lse_strides(t, n: int):
    """Element strides of the leading n dims of an fp32 lse tensor with contiguous rows."""
    import torch
    assert t.dtype == torch.float32, "lse must be float32"
    return _strides(t, n)


def _stream(stream) -> int:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def kvec_workspace_size(cfg: Config) -> int:
    out = ctypes.c_size_t(0)
    c = cfg.c()
    _check(load().kvec_workspace_size(ctypes.byref(c), ctypes.byref(out)), "kvec_workspace_size")
    return out.value


def kvec_score(cfg: Config, q_win, k, p_raw, p_ext_raw, imp, ws, stream=None) -> None:
    """q_win [b][HQ][O'][d], k [b][H][T][d]; outputs fp32 [b][H][Tc], [b][H][Tc], [b][Tc]."""
    c = cfg.c()
    _check(load().kvec_score(ctypes.byref(c), _ptr(q_win), _strides(q_win, 3), _ptr(k),
                             _strides(k, 3), _ptr(p_raw), _ptr(p_ext_raw), _ptr(imp), _ptr(ws),
                             ws.numel() * ws.element_size(), _stream(stream)), "kvec_score")


def kvec_score_lse(cfg: Config, q_win, lse, k, p_raw, p_ext_raw, imp, ws, stream=None) -> None:
    """As kvec_score, with the window rows' natural-log normalisers lse fp32 [b][HQ][O']."""
    c = cfg.c()
    _check(load().kvec_score_lse(ctypes.byref(c), _ptr(q_win), _strides(q_win, 3), _ptr(lse),
                                 _lse_strides(lse, 2), _ptr(k), _strides(k, 3), _ptr(p_raw),
                                 _ptr(p_ext_raw), _ptr(imp), _ptr(ws),
                                 ws.numel() * ws.element_size(), _stream(stream)), "kvec_score_lse")


def kvec_select_cover(cfg: Config, layer: int, p_raw, p_ext_raw, imp, cover_bits, idx,
                      htop_mask=None, ws=None, stream=None) -> None:
    c = cfg.c()
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load().kvec_select_cover(ctypes.byref(c), layer, _ptr(p_raw), _ptr(p_ext_raw), _ptr(imp),
                                    _ptr(cover_bits), _ptr(idx), _ptr(htop_mask), _ptr(ws), nbytes,
                                    _stream(stream)), "kvec_select_cover")


def kvec_compact(cfg: Config, k, v, idx, k_out, v_out, stream=None) -> None:
    c = cfg.c()
    _check(load().kvec_compact(ctypes.byref(c), _ptr(k), _strides(k, 3), _ptr(v), _strides(v, 3),
                               _ptr(idx), _ptr(k_out), _ptr(v_out), _stream(stream)), "kvec_compact")


def kvec_evict_layer(cfg: Config, layer: int, q_win, k, v, cover_bits, idx, k_out, v_out, ws,
                     stream=None) -> None:
    c = cfg.c()
    _check(load().kvec_evict_layer(ctypes.byref(c), layer, _ptr(q_win), _strides(q_win, 3), _ptr(k),
                                   _strides(k, 3), _ptr(v), _strides(v, 3), _ptr(cover_bits),
                                   _ptr(idx), _ptr(k_out), _ptr(v_out), _ptr(ws),
                                   ws.numel() * ws.element_size(), _stream(stream)),
           "kvec_evict_layer")


def kvec_evict_model(cfg: Config, q_win, k, v, cover_bits, idx, k_out, v_out, ws, stream=None,
                     events=None) -> None:
    """q_win [L][b][HQ][O'][d], k/v [L][b][H][T][d]; idx [L][b][H][B]; k_out/v_out [L][b][H][B][d].
    events: optional sequence of kvec_profile_points(cfg) raw hipEvent_t handles (ints)."""
    c = cfg.c()
    ev = None
    if events is not None:
        ev = (ctypes.c_void_p * len(events))(*events)
    _check(load().kvec_evict_model(ctypes.byref(c), _ptr(q_win), _strides(q_win, 4), _ptr(k),
                                   _strides(k, 4), _ptr(v), _strides(v, 4), _ptr(cover_bits),
                                   _ptr(idx), _ptr(k_out), _ptr(v_out), _ptr(ws),
                                   ws.numel() * ws.element_size(), _stream(stream), ev),
           "kvec_evict_model")


def kvec_evict_model_steps(cfg: Config, q_win, k, v, cover_bits, idx, k_out, v_out, ws,
                           stream=None) -> None:
    """n independent steps in one pipelined call: q_win [n][L][b][HQ][O'][d], k/v
    [n][L][b][H][T][d] (any element strides, a step stride of 0 included);
    cover_bits [n][b][L][W], idx [n][L][b][H][B], k_out/v_out [n][L][b][H][B][d]
    contiguous."""
    c = cfg.c()
    n = k.shape[0]
    _check(load().kvec_evict_model_steps(ctypes.byref(c), n, _ptr(q_win), _strides(q_win, 5), _ptr(k),
                                         _strides(k, 5), _ptr(v), _strides(v, 5), _ptr(cover_bits),
                                         _ptr(idx), _ptr(k_out), _ptr(v_out), _ptr(ws),
                                         ws.numel() * ws.element_size(), _stream(stream)),
           "kvec_evict_model_steps")


def kvec_evict_model_lse_steps(cfg: Config, q_win, lse, k, v, cover_bits, idx, k_out, v_out, ws,
                               stream=None) -> None:
    """As kvec_evict_model_steps, with the window rows' natural-log normalisers
    lse fp32 [n][L][b][HQ][O'] (any leading strides, rows contiguous)."""
    c = cfg.c()
    n = k.shape[0]
    _check(load().kvec_evict_model_lse_steps(ctypes.byref(c), n, _ptr(q_win), _strides(q_win, 5),
                                             _ptr(lse), _lse_strides(lse, 4), _ptr(k), _strides(k, 5),
                                             _ptr(v), _strides(v, 5), _ptr(cover_bits), _ptr(idx),
                                             _ptr(k_out), _ptr(v_out), _ptr(ws),
                                             ws.numel() * ws.element_size(), _stream(stream)),
           "kvec_evict_model_lse_steps")


def kvec_evict_model_scores(cfg: Config, q_win, k, v, cover_bits, idx, k_out, v_out, p_raw_out,
                            p_ext_out, imp_out, htop_out, ws, stream=None) -> None:
    """As kvec_evict_model, also writing each layer's scores before pooling:
    p_raw_out, p_ext_out fp32 [L][b][H][Tc] (P over O' for the H_top heads only),
    imp_out fp32 [L][b][Tc], htop_out int32/uint32 [L][b] (H_top bit masks)."""
    c = cfg.c()
    _check(load().kvec_evict_model_scores(ctypes.byref(c), _ptr(q_win), _strides(q_win, 4),
                                          _ptr(k), _strides(k, 4), _ptr(v), _strides(v, 4),
                                          _ptr(cover_bits), _ptr(idx), _ptr(k_out), _ptr(v_out),
                                          _ptr(p_raw_out), _ptr(p_ext_out), _ptr(imp_out),
                                          _ptr(htop_out), _ptr(ws),
                                          ws.numel() * ws.element_size(), _stream(stream)),
           "kvec_evict_model_scores")


def kvec_evict_layer_lse(cfg: Config, layer: int, q_win, lse, k, v, cover_bits, idx, k_out, v_out,
                         ws, stream=None) -> None:
    """As kvec_evict_layer, with the layer's natural-log row normalisers lse fp32 [b][HQ][O']."""
    c = cfg.c()
    _check(load().kvec_evict_layer_lse(ctypes.byref(c), layer, _ptr(q_win), _strides(q_win, 3),
                                       _ptr(lse), _lse_strides(lse, 2), _ptr(k), _strides(k, 3),
                                       _ptr(v), _strides(v, 3), _ptr(cover_bits), _ptr(idx),
                                       _ptr(k_out), _ptr(v_out), _ptr(ws),
                                       ws.numel() * ws.element_size(), _stream(stream)),
           "kvec_evict_layer_lse")


def kvec_evict_model_lse(cfg: Config, q_win, lse, k, v, cover_bits, idx, k_out, v_out, ws,
                         stream=None, events=None) -> None:
    """As kvec_evict_model, with the window rows' natural-log normalisers lse fp32
    [L][b][HQ][O'] (events: kvec_profile_points_lse(cfg) handles)."""
    c = cfg.c()
    ev = None
    if events is not None:
        ev = (ctypes.c_void_p * len(events))(*events)
    _check(load().kvec_evict_model_lse(ctypes.byref(c), _ptr(q_win), _strides(q_win, 4), _ptr(lse),
                                       _lse_strides(lse, 3), _ptr(k), _strides(k, 4), _ptr(v),
                                       _strides(v, 4), _ptr(cover_bits), _ptr(idx), _ptr(k_out),
                                       _ptr(v_out), _ptr(ws), ws.numel() * ws.element_size(),
                                       _stream(stream), ev),
           "kvec_evict_model_lse")


def kvec_profile_points_lse(cfg: Config) -> int:
    c = cfg.c()
    return int(load().kvec_profile_points_lse(ctypes.byref(c)))


def kvec_profile_points(cfg: Config) -> int:
    c = cfg.c()
    return int(load().kvec_profile_points(ctypes.byref(c)))


def kvec_coverage(cfg: Config, cover_bits, upto_layer: int, count, stream=None) -> None:
    c = cfg.c()
    _check(load().kvec_coverage(ctypes.byref(c), _ptr(cover_bits), upto_layer, _ptr(count),
                                _stream(stream)), "kvec_coverage")


def kvec_decode_workspace_size(cfg: Config, n_ctx: int) -> int:
    out = ctypes.c_size_t(0)
    c = cfg.c()
    _check(load().kvec_decode_workspace_size(ctypes.byref(c), n_ctx, ctypes.byref(out)),
           "kvec_decode_workspace_size")
    return out.value


def kvec_decode_attention(cfg: Config, q, k_cache, v_cache, out, ws, idx=None, n_ctx=None,
                          stream=None) -> None:
    """q [b][HQ][d]; k_cache/v_cache [b][H][n_ctx][d] (rows contiguous); out fp32 [b][HQ][d]."""
    c = cfg.c()
    n = k_cache.shape[2] if n_ctx is None else n_ctx
    assert k_cache.stride()[:2] == v_cache.stride()[:2], "K and V caches share their strides"
    assert k_cache.stride(2) == k_cache.shape[3] and v_cache.stride(2) == v_cache.shape[3], \
        "cache rows must be contiguous"
    _check(load().kvec_decode_attention(ctypes.byref(c), _ptr(q), _strides(q, 2), _ptr(k_cache),
                                        _ptr(v_cache), _strides(k_cache, 2), n, _ptr(idx),
                                        _ptr(out), _ptr(ws), ws.numel() * ws.element_size(),
                                        _stream(stream)), "kvec_decode_attention")


def kvec_decode_attention_noalloc(cfg: Config, q, k_cache, v_cache, out, idx=None, n_ctx=None,
                                  stream=None) -> None:
    """kvec_decode_attention without a workspace: the partial states use the
    library's fixed 4 MiB device scratch (calls overlapping on one device race)."""
    c = cfg.c()
    n = k_cache.shape[2] if n_ctx is None else n_ctx
    assert k_cache.stride()[:2] == v_cache.stride()[:2], "K and V caches share their strides"
    assert k_cache.stride(2) == k_cache.shape[3] and v_cache.stride(2) == v_cache.shape[3], \
        "cache rows must be contiguous"
    _check(load().kvec_decode_attention_noalloc(ctypes.byref(c), _ptr(q), _strides(q, 2),
                                                _ptr(k_cache), _ptr(v_cache), _strides(k_cache, 2),
                                                n, _ptr(idx), _ptr(out), _stream(stream)),
           "kvec_decode_attention_noalloc")
