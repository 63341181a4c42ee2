"""Plain, slow reference of the K-VEC prefill-time eviction step (float64).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library; both consume the same seeded inputs (module ``synth``).

Source: "Coverage-Driven KV Cache Eviction for Efficient and Improved Inference
of LLM" (K-VEC).  Each function names the passage it follows:

* windowed eviction score P                      Sec. 4.1, Eq. (eviction)
* row normaliser (log-sum-exp) of the window rows  Sec. 4.1, Eq. (eviction): the
  softmax denominator of A; eviction runs inside each layer's prefill (Sec. 5.1)
* top-B selection per head, cache store           Sec. 4.1 (equation after Eq. eviction)
* head focus sigma = std of P over tokens         Sec. 4.1
* H_top = delta heads with the LOWEST sigma,
  their P recomputed over the extended window O'  Sec. 4.1; Algorithm 1
* alternative head criterion: entropy             Sec. 5.4 (head-selection ablation)
* coverage = n_t / (l + 1)                        Sec. 4.2
* global importance I = mean over the window of
  the max over heads of A                         Sec. 4.2
* focus = I * (1 - coverage); P' = P + lambda*focus  Sec. 4.2; Algorithm 1
* top beta*B tokens of P per head get P' = 1.0     Sec. 4.2; Algorithm 1
* coverage C = number of unique kept tokens       Sec. 3.2
* decode attention over the kept K/V              Sec. 4.1 (the cache serves decoding)

Readings where the paper is silent (each is listed in the design notes):
heads are KV heads and A of a KV head is the mean over its query heads (GQA);
the causal softmax uses scale 1/sqrt(d) over keys 0..p; the observation window
[T-O, T) is always kept and the top-(B-O) prefix tokens are chosen from [0, T-O);
scores are max-pooled along t (kernel k, stride 1, truncated at the ends) before
sigma, the preserve set and P'; sigma is the population std; ties rank lower
token index (or lower head index) first; the preserve set uses P after the
H_top replacement, per head, K = min(floor(beta*B), B-O); layers are 0-based
and n_t counts earlier layers that kept t in at least one head; the cross-layer
arithmetic is done in fp32, one rounding per operation, on fp32 scores.

Parity pins: every function here is pinned in tests/test_oracle_pins.py
against closed forms, brute force on tiny inputs or invariants.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

__all__ = [
    "window_attention", "window_lse", "window_scores", "to_f32", "maxpool1d", "head_sigma",
    "head_entropy", "focus_heads", "decode_attention",
    "adjusted_heads", "rank_first", "preserve_count", "adjusted_priority",
    "LayerResult", "select_layer", "evict_layer_from_scores", "score_layer",
    "gather_rows", "coverage_count", "counts_from_bits", "layer_bits",
]


# ---------------------------------------------------------------------------
# S1  window scores (Sec. 4.1 Eq. eviction; Sec. 4.1 extended window; Sec. 4.2 I)
# ---------------------------------------------------------------------------

def window_attention(q_win: np.ndarray, k: np.ndarray) -> np.ndarray:
    """Causal softmax attention of the last Wn query rows over all T keys.

    q_win: [H_q][Wn][d] float64, the query rows at positions T-Wn .. T-1.
    k:     [H_kv][T][d] float64.
    Returns Abar [H_kv][Wn][T]: the attention A of each query head (scale
    1/sqrt(d), row at position p sees keys 0..p), averaged over the G query
    heads that share a KV head (query head j uses KV head j // G).
    """
    hq, wn, d = q_win.shape
    hkv, T, _ = k.shape
    g = hq // hkv
    pos = T - wn + np.arange(wn)                     # absolute position of each row
    visible = np.arange(T)[None, :] <= pos[:, None]  # [Wn][T] causal mask
    out = np.zeros((hkv, wn, T))
    for h in range(hkv):
        for jj in range(g):
            j = h * g + jj
            s = (q_win[j] @ k[h].T) / math.sqrt(d)   # [Wn][T] logits
            s = np.where(visible, s, -np.inf)
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            a = e / e.sum(axis=1, keepdims=True)
            out[h] += a
        out[h] /= g
    return out


def window_lse(q_win: np.ndarray, k: np.ndarray) -> np.ndarray:
    """Natural-log softmax normaliser of every window row of every query head.

    q_win: [H_q][Wn][d] float64 (positions T-Wn .. T-1), k: [H_kv][T][d].
    Returns lse [H_q][Wn]: lse[j, r] = ln sum_{t <= p_r} exp(q_{j,r} . k_{j//G,t} / sqrt(d)),
    the denominator of the causal softmax A in the eviction score (Sec. 4.1),
    i.e. the log-sum-exp that the layer's prefill attention produces for
    those query rows.
    """
    hq, wn, d = q_win.shape
    hkv, T, _ = k.shape
    g = hq // hkv
    pos = T - wn + np.arange(wn)
    visible = np.arange(T)[None, :] <= pos[:, None]
    out = np.zeros((hq, wn))
    for j in range(hq):
        s = (q_win[j] @ k[j // g].T) / math.sqrt(d)
        s = np.where(visible, s, -np.inf)
        m = s.max(axis=1)
        out[j] = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
    return out


def window_scores(q_win: np.ndarray, k: np.ndarray, window: int, full: bool = False):
    """P, P over the extended window, and I for one (sequence, layer).

    The rows of q_win are the extended window (O' = Wn rows); the last `window`
    (= O) of them form the observation window.

      P[h,t]     = (1/O)  * sum over the last O rows  of Abar[h,r,t]   (Eq. eviction)
      P_ext[h,t] = (1/O') * sum over all O' rows      of Abar[h,r,t]   (Sec. 4.1)
      I[t]       = (1/O)  * sum over the last O rows  of max_h Abar[h,r,t]  (Sec. 4.2)

    Returned for the candidate tokens t < T - O (all T tokens if full=True).
    """
    abar = window_attention(q_win, k)
    hkv, wn, T = abar.shape
    O = window
    base = abar[:, wn - O:, :]
    p = base.sum(axis=1) / O
    p_ext = abar.sum(axis=1) / wn
    imp = base.max(axis=0).sum(axis=0) / O
    if not full:
        tc = T - O
        p, p_ext, imp = p[:, :tc], p_ext[:, :tc], imp[:tc]
    return p, p_ext, imp


def to_f32(x: np.ndarray) -> np.ndarray:
    """Round float64 to float32, nearest-even (the oracle's fp32 scores)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32)


# ---------------------------------------------------------------------------
# S2  pooling along the token axis (inherited from the SnapKV setting)
# ---------------------------------------------------------------------------

def maxpool1d(x: np.ndarray, kernel: int) -> np.ndarray:
    """pooled[t] = max{ x[u] : |u - t| <= kernel//2, 0 <= u < n } along the last axis."""
    if kernel <= 1:
        return x.copy()
    r = kernel // 2
    n = x.shape[-1]
    pad = np.full(x.shape[:-1] + (r,), -np.inf, dtype=x.dtype)
    xp = np.concatenate([pad, x, pad], axis=-1)
    out = xp[..., 0:n].copy()
    for o in range(1, kernel):
        np.maximum(out, xp[..., o:o + n], out=out)
    return out


# ---------------------------------------------------------------------------
# S3  cross-head coverage (Sec. 4.1; Algorithm 1)
# ---------------------------------------------------------------------------

def head_sigma(p: np.ndarray) -> np.ndarray:
    """Population standard deviation of each head's scores over tokens, in float64:
    sigma_h = sqrt( (1/N) * sum_t (P[h,t] - mean_h)^2 )."""
    x = np.asarray(p, dtype=np.float64)
    mean = x.sum(axis=1) / x.shape[1]
    return np.sqrt(((x - mean[:, None]) ** 2).sum(axis=1) / x.shape[1])


def head_entropy(p: np.ndarray) -> np.ndarray:
    """Shannon entropy (natural log) of each head's scores taken as a distribution
    over tokens, in float64: H_h = -sum_t q_t ln q_t with q_t = P[h,t] / sum_u P[h,u]
    (0 ln 0 = 0; a head whose scores are all zero has entropy 0)."""
    x = np.asarray(p, dtype=np.float64)
    out = np.zeros(x.shape[0])
    for h in range(x.shape[0]):
        tot = x[h].sum()
        if tot > 0:
            q = x[h][x[h] > 0] / tot
            out[h] = -(q * np.log(q)).sum()
    return out


def focus_heads(pooled: np.ndarray, delta: int, criterion: str = "std") -> np.ndarray:
    """H_top by the paper's criterion (the delta lowest sigma, Sec. 4.1) or by the
    alternative of the head-selection ablation (Sec. 5.4): the delta least focused
    heads by entropy, i.e. the highest entropy.  Ties: lower head index first."""
    if criterion == "std":
        return adjusted_heads(head_sigma(pooled), delta)
    if criterion == "entropy":
        return adjusted_heads(-head_entropy(pooled), delta)
    raise ValueError(criterion)


def adjusted_heads(sigma: np.ndarray, delta: int) -> np.ndarray:
    """H_top: the delta heads with the lowest sigma (ties: lower head index first)."""
    order = sorted(range(len(sigma)), key=lambda h: (float(sigma[h]), h))
    return np.array(sorted(order[:max(0, min(delta, len(sigma)))]), dtype=np.int64)


# ---------------------------------------------------------------------------
# S4 / S6  ranking (Sec. 4.1 top-B; Sec. 4.2 preserve set)
# ---------------------------------------------------------------------------

def rank_first(scores: np.ndarray, k: int) -> np.ndarray:
    """Indices of the first k tokens in the order (score descending, index ascending)."""
    n = scores.shape[0]
    k = max(0, min(k, n))
    order = np.lexsort((np.arange(n), -np.asarray(scores, dtype=np.float64)))
    return order[:k]


def preserve_count(budget: int, window: int, beta: float) -> int:
    """K = beta * B tokens preserved per head (Sec. 4.2), capped at the B - O prefix picks."""
    return int(min(math.floor(float(np.float32(beta)) * budget), budget - window))


# ---------------------------------------------------------------------------
# S5  cross-layer coverage bonus (Sec. 4.2; Algorithm 1), fp32 op by op
# ---------------------------------------------------------------------------

def adjusted_priority(p_sel: np.ndarray, imp: np.ndarray, n_t: np.ndarray, layer: int,
                      lam: float, keep: np.ndarray) -> np.ndarray:
    """P' = P + lambda * I * (1 - n_t / (l + 1)), then P' = 1.0 on the preserved set.

    p_sel: [H][Tc] fp32 (after pooling and the H_top replacement); imp: [Tc] fp32;
    n_t: [Tc] integer counts; keep: [H][Tc] bool.  Every operation is one fp32
    operation rounded to nearest-even (numpy float32 arithmetic, no fusion)."""
    f32 = np.float32
    cov = n_t.astype(f32) / f32(layer + 1)          # coverage_{l,t}
    focus = imp.astype(f32) * (f32(1.0) - cov)       # focus_{l,t}
    bonus = f32(lam) * focus                         # lambda * focus, broadcast over heads
    out = p_sel.astype(f32) + bonus[None, :]
    out[keep] = f32(1.0)
    return out


# ---------------------------------------------------------------------------
# One layer of the policy on given fp32 scores (S2 .. S7)
# ---------------------------------------------------------------------------

@dataclass
class LayerResult:
    idx: np.ndarray        # [H][B] int32 kept token indices (ascending prefix picks, then window); -1 pads
    htop: np.ndarray       # sorted head indices whose P was replaced by P_ext
    sigma: np.ndarray      # [H] float64
    keep: np.ndarray       # [H][Tc] bool, the preserved set
    p_sel: np.ndarray      # [H][Tc] fp32, pooled P after the H_top replacement
    p_adj: np.ndarray      # [H][Tc] fp32, P'
    bits: np.ndarray       # [T] bool, kept by at least one head at this layer


def select_layer(p_raw: np.ndarray, p_ext_raw: np.ndarray, imp: np.ndarray, n_t: np.ndarray,
                 layer: int, *, T: int, window: int, window_ext: int, budget: int,
                 pool_kernel: int, delta: int, lam: float, beta: float,
                 criterion: str = "std") -> LayerResult:
    """The per-layer K-VEC policy on fp32 scores (Algorithm 1, then top-B and the window).

    p_raw, p_ext_raw: [H][Tc] fp32; imp: [Tc] fp32; n_t: [T] (or [Tc]) layer counts."""
    H = p_raw.shape[0]
    O = window
    Tc = T - O
    if T <= budget:                                  # nothing to evict
        idx = np.full((H, budget), -1, dtype=np.int32)
        idx[:, :T] = np.arange(T, dtype=np.int32)[None, :]
        z = np.zeros((H, max(Tc, 0)), dtype=bool)
        return LayerResult(idx, np.zeros(0, np.int64), np.zeros(H), z,
                           np.zeros((H, max(Tc, 0)), np.float32), np.zeros((H, max(Tc, 0)), np.float32),
                           np.ones(T, dtype=bool))
    pooled = maxpool1d(p_raw.astype(np.float32), pool_kernel)
    pooled_ext = maxpool1d(p_ext_raw.astype(np.float32), pool_kernel)
    sigma = head_sigma(pooled)
    wn = min(window_ext, T)
    htop = focus_heads(pooled, delta, criterion) if wn > O else np.zeros(0, np.int64)
    p_sel = pooled.copy()
    p_sel[htop] = pooled_ext[htop]
    kp = preserve_count(budget, O, beta)
    keep = np.zeros((H, Tc), dtype=bool)
    for h in range(H):
        keep[h, rank_first(p_sel[h], kp)] = True
    p_adj = adjusted_priority(p_sel, imp, np.asarray(n_t)[:Tc], layer, lam, keep)
    m = budget - O
    idx = np.empty((H, budget), dtype=np.int32)
    bits = np.zeros(T, dtype=bool)
    bits[Tc:] = True
    for h in range(H):
        pick = np.sort(rank_first(p_adj[h], m))
        idx[h, :m] = pick
        idx[h, m:] = np.arange(Tc, T)
        bits[pick] = True
    return LayerResult(idx, htop, sigma, keep, p_sel, p_adj, bits)


def evict_layer_from_scores(p_raw, p_ext_raw, imp, n_t, layer, w) -> LayerResult:
    """select_layer with the hyper-parameters of a workload description `w`."""
    return select_layer(p_raw, p_ext_raw, imp, n_t, layer, T=w.seq_len, window=w.window,
                        window_ext=w.window_ext, budget=w.budget, pool_kernel=w.pool_kernel,
                        delta=w.n_adjust_heads, lam=w.lam, beta=w.beta,
                        criterion=getattr(w, "criterion", "std"))


def score_layer(q_win: np.ndarray, k: np.ndarray, window: int):
    """Oracle scores of one (sequence, layer): float64 P, P_ext, I rounded to fp32."""
    p, pe, imp = window_scores(q_win, k, window)
    return to_f32(p), to_f32(pe), to_f32(imp)


# ---------------------------------------------------------------------------
# S7  coverage state; S8  cache store
# ---------------------------------------------------------------------------

def counts_from_bits(layer_bits_list) -> np.ndarray:
    """n_t = number of earlier layers whose kept set (over all heads) contains t."""
    if len(layer_bits_list) == 0:
        return None
    return np.sum(np.stack([np.asarray(b, dtype=np.int64) for b in layer_bits_list]), axis=0)


def layer_bits(idx: np.ndarray, T: int) -> np.ndarray:
    """Tokens kept by at least one head: the union of a layer's index sets."""
    bits = np.zeros(T, dtype=bool)
    v = idx[idx >= 0]
    bits[v] = True
    return bits


def coverage_count(layer_bits_list) -> int:
    """Coverage C = number of unique tokens kept across all heads and layers (Sec. 3.2)."""
    u = np.zeros_like(np.asarray(layer_bits_list[0], dtype=bool))
    for b in layer_bits_list:
        u |= np.asarray(b, dtype=bool)
    return int(u.sum())


def gather_rows(x: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """Cache store: out[h][i] = x[h][idx[h][i]] (zeros where idx is -1)."""
    H, B = idx.shape
    out = np.zeros((H, B) + x.shape[2:], dtype=x.dtype)
    for h in range(H):
        ok = idx[h] >= 0
        out[h, ok] = x[h, idx[h, ok]]
    return out


# ---------------------------------------------------------------------------
# After the step: one decode token's attention over the compacted cache
# ---------------------------------------------------------------------------

def decode_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, valid=None) -> np.ndarray:
    """Softmax attention of one new token over the kept cache rows (float64).

    q: [H_q][d]; k, v: [H_kv][n][d]; valid: [H_kv][n] bool or None (all rows).
    out[j] = sum_i softmax_i(q_j . k_{j//G,i} / sqrt(d)) v_{j//G,i} over the
    valid rows i of KV head j // G; a head with no valid row gives zeros."""
    hq, d = q.shape
    hkv = k.shape[0]
    g = hq // hkv
    out = np.zeros((hq, d))
    for j in range(hq):
        h = j // g
        rows = np.arange(k.shape[1]) if valid is None else np.nonzero(valid[h])[0]
        if len(rows) == 0:
            continue
        s = (k[h, rows] @ q[j]) / math.sqrt(d)
        e = np.exp(s - s.max())
        out[j] = (e / e.sum()) @ v[h, rows]
    return out
