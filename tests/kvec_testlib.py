"""Shared helpers of the GPU parity tests: seeded inputs on the device, the
oracle on the same bytes, and the agreement / tolerance checks."""
from __future__ import annotations

import numpy as np

import oracle as orc
import synth

SCORE_RTOL = 2e-3      # score relative error bound (bf16 inputs, fp32 accumulation)
AGREE_MIN = 0.995      # end-to-end index agreement
CUT_RTOL = 4e-3        # a mismatch must sit within this of the cut (two score errors)


def torch_dtype(w):
    import torch
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


def to_device(a: np.ndarray, w):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a))
    if w.dtype == "bf16":
        t = t.view(torch.bfloat16)
    return t.cuda()


def layer_inputs(w, layer: int, b: int):
    """Host arrays of one (layer, sequence): q [HQ][Wn][d], k/v [H][T][d] (storage dtype)."""
    return synth.queries(w, layer, b), synth.keys(w, layer, b), synth.values(w, layer, b)


def model_tensors(w, layers=None):
    """Device tensors q [L][b][HQ][Wn][d], k/v [L][b][H][T][d] for the whole workload."""
    import torch
    L = w.n_layers if layers is None else layers
    dt = torch_dtype(w)
    q = torch.empty((L, w.batch, w.n_q_heads, w.rows, w.head_dim), dtype=dt, device="cuda")
    k = torch.empty((L, w.batch, w.n_kv_heads, w.seq_len, w.head_dim), dtype=dt, device="cuda")
    v = torch.empty_like(k)
    for l in range(L):
        for b in range(w.batch):
            qa, ka, va = layer_inputs(w, l, b)
            q[l, b].copy_(to_device(qa, w))
            k[l, b].copy_(to_device(ka, w))
            v[l, b].copy_(to_device(va, w))
    return q, k, v


def oracle_scores(w, layer: int, b: int, q=None, k=None):
    """Oracle fp32 scores (float64 computation on the exact input values)."""
    if q is None:
        q = synth.queries(w, layer, b)
        k = synth.keys(w, layer, b)
    qf = synth.to_f64(q, w.dtype)
    kf = synth.to_f64(k, w.dtype)
    p, pe, imp = orc.window_scores(qf, kf, w.window)
    return p, pe, imp


def rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.max(np.abs(got - ref) / np.maximum(np.abs(ref), 1e-30)))


def bits_to_bool(words: np.ndarray, T: int) -> np.ndarray:
    """uint64 bitmap row -> bool[T]."""
    u = np.asarray(words, dtype=np.uint64)
    bits = ((u[:, None] >> np.arange(64, dtype=np.uint64)[None, :]) & np.uint64(1)).astype(bool)
    return bits.reshape(-1)[:T]


def counts_before(bits_rows: np.ndarray, layer: int, T: int) -> np.ndarray:
    """n_t from bitmap rows [L][W] of the layers before `layer`."""
    n = np.zeros(T, dtype=np.int64)
    for l in range(layer):
        n += bits_to_bool(bits_rows[l], T)
    return n


def agreement(gpu_idx: np.ndarray, res: orc.LayerResult, M: int, kp: int):
    """Teacher-forced comparison of one layer for one sequence.

    Returns (matched, total, bad) where `bad` lists mismatched tokens that are
    NOT within CUT_RTOL of the oracle's cut (of P' for the final pick, or of
    P_sel for the preserve set)."""
    H = gpu_idx.shape[0]
    matched, total, bad = 0, 0, []
    for h in range(H):
        g = set(int(x) for x in gpu_idx[h, :M])
        o = set(int(x) for x in res.idx[h, :M])
        matched += len(g & o)
        total += M
        if g == o:
            continue
        padj = res.p_adj[h].astype(np.float64)
        cut = np.sort(padj)[::-1][M - 1]
        psel = res.p_sel[h].astype(np.float64)
        kcut = np.sort(psel)[::-1][kp - 1] if kp > 0 else None
        for t in g ^ o:
            near_cut = abs(padj[t] - cut) <= CUT_RTOL * abs(cut)
            near_keep = kcut is not None and abs(psel[t] - kcut) <= CUT_RTOL * abs(kcut)
            if not (near_cut or near_keep):
                bad.append((h, t, float(padj[t]), float(cut)))
    return matched, total, bad
