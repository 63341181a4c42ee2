"""Pins of the CPU oracle to facts fixed by the paper and by mathematics.

Each check is written once as a function of the oracle routine(s) it pins, so
that the mutation tests at the end can plant a plausible mistake in a copy of
the oracle and show that the same check fails.  Nothing here calls the GPU.
"""
import math
import statistics

import numpy as np
import pytest

import oracle as orc


def _rng(seed):
    return np.random.default_rng(seed)


def _harmonic(n):
    return math.fsum(1.0 / i for i in range(1, n + 1))


# --------------------------------------------------------------------------
# S1: window scores
# --------------------------------------------------------------------------

def check_zero_query_closed_form(window_scores):
    """Q = 0: every visible logit is 0, so row r at position p has A = 1/(p+1).
    P[t]  = (H_T - H_{T-O}) / O for every candidate t (all base rows see t);
    P'[t] = (H_T - H_{max(t, T-O')}) / O'  (causal edge of the extended window);
    I[t]  = P[t] (every head is identical).  H_n is the n-th harmonic number."""
    T, wn, O, hkv, g, d = 53, 10, 4, 3, 2, 8
    k = _rng(1).standard_normal((hkv, T, d))
    q = np.zeros((hkv * g, wn, d))
    p, pe, imp = window_scores(q, k, O)
    Tc = T - O
    want_p = (_harmonic(T) - _harmonic(T - O)) / O
    want_pe = np.array([(_harmonic(T) - _harmonic(max(t, T - wn))) / wn for t in range(Tc)])
    assert p.shape == (hkv, Tc) and pe.shape == (hkv, Tc) and imp.shape == (Tc,)
    np.testing.assert_allclose(p, want_p, rtol=1e-13, atol=0)
    np.testing.assert_allclose(pe, np.broadcast_to(want_pe, pe.shape), rtol=1e-13, atol=0)
    np.testing.assert_allclose(imp, want_p, rtol=1e-13, atol=0)


def _brute_scores(q, k, O):
    """Pure-Python loops: causal softmax per query head, mean over the G heads of a
    KV head, window sums, max over KV heads.  Shares nothing with the oracle."""
    hq, wn, d = len(q), len(q[0]), len(q[0][0])
    hkv, T = len(k), len(k[0])
    g = hq // hkv
    abar = [[[0.0] * T for _ in range(wn)] for _ in range(hkv)]
    for j in range(hq):
        h = j // g
        for r in range(wn):
            p = T - wn + r
            logits = [math.fsum(q[j][r][i] * k[h][t][i] for i in range(d)) / math.sqrt(d)
                      for t in range(p + 1)]
            mx = max(logits)
            ex = [math.exp(x - mx) for x in logits]
            z = math.fsum(ex)
            for t in range(p + 1):
                abar[h][r][t] += ex[t] / z / g
    Tc = T - O
    P = [[math.fsum(abar[h][r][t] for r in range(wn - O, wn)) / O for t in range(Tc)]
         for h in range(hkv)]
    PE = [[math.fsum(abar[h][r][t] for r in range(wn)) / wn for t in range(Tc)] for h in range(hkv)]
    I = [math.fsum(max(abar[h][r][t] for h in range(hkv)) for r in range(wn - O, wn)) / O
         for t in range(Tc)]
    return np.array(P), np.array(PE), np.array(I)


def check_brute_force(window_scores):
    for seed, (T, wn, O, hkv, g, d) in enumerate([(17, 5, 2, 2, 2, 4), (23, 7, 3, 3, 1, 6),
                                                  (12, 12, 4, 2, 3, 4), (9, 4, 4, 1, 4, 2)]):
        r = _rng(100 + seed)
        q = r.standard_normal((hkv * g, wn, d)) * 2.0
        k = r.standard_normal((hkv, T, d)) * 2.0
        p, pe, imp = window_scores(q, k, O)
        bp, bpe, bimp = _brute_scores(q.tolist(), k.tolist(), O)
        np.testing.assert_allclose(p, bp, rtol=1e-11, atol=1e-300)
        np.testing.assert_allclose(pe, bpe, rtol=1e-11, atol=1e-300)
        np.testing.assert_allclose(imp, bimp, rtol=1e-11, atol=1e-300)


def check_mass(window_scores):
    """Each query row's attention sums to 1, so over all T tokens P and P' sum to 1."""
    r = _rng(7)
    q = r.standard_normal((8, 12, 16)) * 3
    k = r.standard_normal((4, 300, 16))
    p, pe, imp = window_scores(q, k, 5, full=True)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(pe.sum(axis=1), 1.0, rtol=1e-13)
    assert np.all(imp >= p.max(axis=0) * (1 - 1e-14))   # max over heads >= each head


def check_identical_heads(window_scores):
    """All KV heads (and their query groups) identical: I equals every head's P."""
    r = _rng(9)
    k1 = r.standard_normal((1, 64, 8))
    q1 = r.standard_normal((2, 6, 8))
    k = np.repeat(k1, 3, axis=0)
    q = np.concatenate([q1] * 3, axis=0)
    p, pe, imp = window_scores(q, k, 3)
    for h in range(3):
        np.testing.assert_allclose(p[h], imp, rtol=1e-14)
    p1, _, imp1 = window_scores(q1, k1, 3)
    np.testing.assert_allclose(imp1, p1[0], rtol=1e-14)


def check_single_row_softmax(window_scores):
    """O = O' = 1 and G = 1: P is the plain softmax of the last row over t < T-1."""
    r = _rng(11)
    q = r.standard_normal((1, 1, 8))
    k = r.standard_normal((1, 40, 8))
    p, pe, imp = window_scores(q, k, 1)
    s = (k[0] @ q[0, 0]) / math.sqrt(8)
    e = np.exp(s - s.max())
    sm = e / e.sum()
    np.testing.assert_allclose(p[0], sm[:39], rtol=1e-13)
    np.testing.assert_allclose(pe[0], sm[:39], rtol=1e-13)


def check_lse_constant_keys(window_lse):
    """Every key of KV head h equal to c_h: every visible logit of row r of query
    head j is s = q_{j,r} . c_{j//G} / sqrt(d), and row r at position p sees p+1
    keys, so lse = s + ln(p + 1).  Distinct c_h pin the query-to-KV-head map."""
    T, wn, hkv, g, d = 40, 6, 3, 2, 8
    r = _rng(21)
    c = r.standard_normal((hkv, d))
    k = np.repeat(c[:, None, :], T, axis=1)
    q = r.standard_normal((hkv * g, wn, d))
    lse = window_lse(q, k)
    assert lse.shape == (hkv * g, wn)
    for j in range(hkv * g):
        for row in range(wn):
            s = float(q[j, row] @ c[j // g]) / math.sqrt(d)
            want = s + math.log(T - wn + row + 1)
            assert abs(lse[j, row] - want) <= 1e-12 * max(1.0, abs(want)), (j, row)


def check_lse_brute(window_lse):
    """Pure-Python loops, log of the fsum of exps over the causal keys."""
    for seed, (T, wn, hkv, g, d) in enumerate([(15, 5, 2, 2, 4), (9, 9, 1, 3, 6)]):
        r = _rng(300 + seed)
        q = r.standard_normal((hkv * g, wn, d)) * 2.0
        k = r.standard_normal((hkv, T, d)) * 2.0
        lse = window_lse(q, k)
        for j in range(hkv * g):
            for row in range(wn):
                p = T - wn + row
                z = math.fsum(math.exp(math.fsum(q[j, row, i] * k[j // g, t, i] for i in range(d))
                                       / math.sqrt(d)) for t in range(p + 1))
                assert abs(lse[j, row] - math.log(z)) <= 1e-12 * max(1.0, abs(math.log(z)))


def check_lse_normalises_scores(window_lse):
    """One row, one head: exp(logit - lse) over the candidates is the score P of
    window_scores (O = O' = 1), which the mass identity pins independently."""
    r = _rng(22)
    q = r.standard_normal((1, 1, 8)) * 3
    k = r.standard_normal((1, 50, 8))
    lse = window_lse(q, k)
    p, _, _ = orc.window_scores(q, k, 1)
    s = (k[0, :49] @ q[0, 0]) / math.sqrt(8)
    np.testing.assert_allclose(np.exp(s - lse[0, 0]), p[0], rtol=1e-12)


def test_lse_constant_keys():
    check_lse_constant_keys(orc.window_lse)


def test_lse_brute_force():
    check_lse_brute(orc.window_lse)


def test_lse_normalises_scores():
    check_lse_normalises_scores(orc.window_lse)


def check_decode_constant_keys(decode_attention):
    """All keys of a head equal: uniform weights, so out = the mean of the valid
    V rows; distinct keys per head pin the query-to-KV-head map through V."""
    r = _rng(25)
    hkv, g, n, d = 2, 3, 11, 8
    k = np.repeat(r.standard_normal((hkv, 1, d)), n, axis=1)
    v = r.standard_normal((hkv, n, d))
    q = r.standard_normal((hkv * g, d))
    valid = np.ones((hkv, n), bool)
    valid[1, [0, 4, 5]] = False
    out = decode_attention(q, k, v, valid)
    for j in range(hkv * g):
        want = v[j // g][valid[j // g]].mean(axis=0)
        np.testing.assert_allclose(out[j], want, rtol=1e-13, atol=1e-15)


def check_decode_brute(decode_attention):
    r = _rng(26)
    hkv, g, n, d = 2, 2, 7, 4
    q = r.standard_normal((hkv * g, d)) * 2
    k = r.standard_normal((hkv, n, d)) * 2
    v = r.standard_normal((hkv, n, d))
    valid = r.random((hkv, n)) > 0.3
    out = decode_attention(q, k, v, valid)
    for j in range(hkv * g):
        h = j // g
        logits = [math.fsum(q[j, i] * k[h, t, i] for i in range(d)) / math.sqrt(d)
                  for t in range(n) if valid[h, t]]
        vs = [v[h, t] for t in range(n) if valid[h, t]]
        mx = max(logits)
        ex = [math.exp(x - mx) for x in logits]
        z = math.fsum(ex)
        for c in range(d):
            want = math.fsum(ex[i] / z * vs[i][c] for i in range(len(vs)))
            assert abs(out[j, c] - want) <= 1e-12


def test_decode_constant_keys():
    check_decode_constant_keys(orc.decode_attention)


def test_decode_brute_force():
    check_decode_brute(orc.decode_attention)


def test_decode_single_row_and_empty():
    r = _rng(27)
    q = r.standard_normal((2, 4))
    k = r.standard_normal((1, 5, 4))
    v = r.standard_normal((1, 5, 4))
    valid = np.zeros((1, 5), bool)
    np.testing.assert_array_equal(orc.decode_attention(q, k, v, valid), 0.0)
    valid[0, 3] = True
    np.testing.assert_allclose(orc.decode_attention(q, k, v, valid), np.stack([v[0, 3]] * 2),
                               rtol=1e-15)


def test_zero_query_closed_form():
    check_zero_query_closed_form(orc.window_scores)


def test_window_scores_brute_force():
    check_brute_force(orc.window_scores)


def test_mass_identity():
    check_mass(orc.window_scores)


def test_identical_heads():
    check_identical_heads(orc.window_scores)


def test_single_row_softmax():
    check_single_row_softmax(orc.window_scores)


def test_head_permutation_equivariance():
    r = _rng(12)
    hkv, g = 4, 2
    q = r.standard_normal((hkv * g, 6, 8))
    k = r.standard_normal((hkv, 50, 8))
    perm = np.array([2, 0, 3, 1])
    qperm = q.reshape(hkv, g, 6, 8)[perm].reshape(hkv * g, 6, 8)
    p, pe, imp = orc.window_scores(q, k, 3)
    p2, pe2, imp2 = orc.window_scores(qperm, k[perm], 3)
    np.testing.assert_allclose(p2, p[perm], rtol=1e-13)
    np.testing.assert_allclose(pe2, pe[perm], rtol=1e-13)
    np.testing.assert_allclose(imp2, imp, rtol=1e-13)


def test_to_f32_round_to_nearest_even():
    x = np.array([1.0 + 2.0 ** -24, 1.0 + 3 * 2.0 ** -24, 1.0 + 2.0 ** -25])
    y = orc.to_f32(x)
    assert y.dtype == np.float32
    assert y[0] == np.float32(1.0)                      # tie -> even
    assert y[1] == np.float32(1.0 + 2.0 ** -22)         # tie -> even (up)
    assert y[2] == np.float32(1.0)


# --------------------------------------------------------------------------
# S2: max pooling
# --------------------------------------------------------------------------

def check_maxpool(maxpool1d):
    r = _rng(13)
    for n, kern in [(1, 7), (5, 7), (20, 5), (33, 7), (10, 1), (9, 3)]:
        x = r.integers(0, 6, size=(2, n)).astype(np.float32)   # many exact ties
        got = maxpool1d(x, kern)
        rad = kern // 2
        want = np.array([[max(x[h, max(0, t - rad):min(n, t + rad + 1)]) for t in range(n)]
                         for h in range(2)], dtype=np.float32)
        np.testing.assert_array_equal(got, want)


def test_maxpool_naive():
    check_maxpool(orc.maxpool1d)


def test_maxpool_identity_kernel_one():
    x = _rng(14).standard_normal((3, 17)).astype(np.float32)
    np.testing.assert_array_equal(orc.maxpool1d(x, 1), x)


# --------------------------------------------------------------------------
# S3: head focus and the adjusted heads
# --------------------------------------------------------------------------

def check_sigma(head_sigma):
    r = _rng(15)
    x = r.random((5, 31)).astype(np.float32)
    got = head_sigma(x)
    for h in range(5):
        want = statistics.pstdev([float(v) for v in x[h]])   # exact rational arithmetic
        assert abs(got[h] - want) <= 1e-15 * max(want, 1e-30) + 1e-17


def check_lowest_sigma(adjusted_heads):
    """H_top holds the delta heads with the LOWEST sigma (Sec. 4.1); ties -> lower head."""
    s = np.array([3.0, 1.0, 2.0, 1.0, 0.5])
    assert list(adjusted_heads(s, 2)) == [1, 4]
    assert list(adjusted_heads(s, 3)) == [1, 3, 4]
    assert list(adjusted_heads(s, 0)) == []
    assert list(adjusted_heads(s, 9)) == [0, 1, 2, 3, 4]


def check_entropy_closed_forms(head_entropy):
    """Uniform scores: ln N.  One non-zero score: 0.  k scores of a and N-k of b:
    with u = k*a + (N-k)*b, H = -(k*a/u) ln(a/u) - ((N-k)*b/u) ln(b/u).  Scaling a
    head's scores does not change its entropy (they are normalised first)."""
    N = 40
    x = np.zeros((4, N), dtype=np.float32)
    x[0] = 0.25
    x[1, 7] = 3.0
    a, b, k = 0.5, 0.125, 9
    x[2, :k] = a
    x[2, k:] = b
    x[3] = x[2] * 8.0
    got = head_entropy(x)
    u = k * a + (N - k) * b
    want2 = -(k * a / u) * math.log(a / u) - ((N - k) * b / u) * math.log(b / u)
    assert abs(got[0] - math.log(N)) <= 1e-14
    assert got[1] == 0.0
    assert abs(got[2] - want2) <= 1e-14
    assert abs(got[3] - want2) <= 1e-14


def check_entropy_brute(head_entropy):
    r = _rng(23)
    x = r.random((3, 57)).astype(np.float32)
    x[1, ::5] = 0.0
    got = head_entropy(x)
    for h in range(3):
        tot = math.fsum(float(v) for v in x[h])
        want = -math.fsum((float(v) / tot) * math.log(float(v) / tot) for v in x[h] if v > 0)
        assert abs(got[h] - want) <= 1e-13


def check_entropy_picks_least_focused(focus_heads):
    """The entropy criterion takes the delta HIGHEST-entropy heads (the least
    focused); sigma and entropy can disagree, so build heads where they do.
    Head 0: uniform; head 1: one spike; head 2: two equal spikes on a floor;
    head 3: a half-and-half two-level head scaled up (large sigma, high entropy)."""
    N = 64
    x = np.full((4, N), 1e-6, dtype=np.float32)
    x[0] = 0.01
    x[1, 3] = 1.0
    x[2, 5] = x[2, 9] = 0.5
    x[3, :32] = 10.0
    x[3, 32:] = 5.0
    ent = orc.head_entropy(x)
    sig = orc.head_sigma(x)
    assert list(np.argsort(-ent, kind="stable")[:2]) == [0, 3]
    assert list(np.argsort(sig, kind="stable")[:2]) == [0, 2]      # sigma disagrees on head 3
    assert list(focus_heads(x, 2, "entropy")) == [0, 3]
    assert list(focus_heads(x, 2, "std")) == [0, 2]
    y = np.stack([x[0], x[0], x[1]])                                  # tie -> lower head
    assert list(focus_heads(y, 1, "entropy")) == [0]


def test_sigma_population_std():
    check_sigma(orc.head_sigma)


def test_entropy_closed_forms():
    check_entropy_closed_forms(orc.head_entropy)


def test_entropy_brute_force():
    check_entropy_brute(orc.head_entropy)


def test_entropy_picks_least_focused():
    check_entropy_picks_least_focused(orc.focus_heads)


def test_entropy_criterion_inert_when_every_head_adjusted():
    """delta = H replaces every head whatever the criterion: same selection."""
    r = _rng(24)
    H, T, O = 4, 300, 8
    p = r.random((H, T - O)).astype(np.float32) * 1e-3
    pe = r.random((H, T - O)).astype(np.float32) * 1e-3
    imp = r.random(T - O).astype(np.float32) * 1e-3
    kw = dict(T=T, window=O, window_ext=16, budget=40, pool_kernel=3, lam=1.0, beta=0.25)
    a = orc.select_layer(p, pe, imp, np.zeros(T, np.int64), 1, delta=H, criterion="std", **kw)
    b = orc.select_layer(p, pe, imp, np.zeros(T, np.int64), 1, delta=H, criterion="entropy", **kw)
    np.testing.assert_array_equal(a.idx, b.idx)


def test_adjusted_heads_lowest_sigma():
    check_lowest_sigma(orc.adjusted_heads)


# --------------------------------------------------------------------------
# S4/S6: ranking
# --------------------------------------------------------------------------

def check_rank_brute(rank_first):
    """Brute force: t is among the first k iff fewer than k tokens precede it in the
    order (score desc, index asc)."""
    r = _rng(16)
    for n in [1, 2, 7, 30, 64]:
        s = r.integers(0, 5, size=n).astype(np.float32)
        for k in [0, 1, n // 2, n]:
            got = set(int(i) for i in rank_first(s, k))
            want = set()
            for t in range(n):
                ahead = sum(1 for u in range(n) if s[u] > s[t] or (s[u] == s[t] and u < t))
                if ahead < k:
                    want.add(t)
            assert got == want, (n, k)
            assert len(rank_first(s, k)) == k


def test_rank_first_brute_force():
    check_rank_brute(orc.rank_first)


def test_preserve_count():
    assert orc.preserve_count(128, 32, 0.25) == 32
    assert orc.preserve_count(1024, 32, 0.25) == 256
    assert orc.preserve_count(512, 64, 0.25) == 128
    assert orc.preserve_count(2048, 32, 0.25) == 512
    assert orc.preserve_count(128, 32, 1.0) == 96       # capped at B - O
    assert orc.preserve_count(128, 32, 0.0) == 0


# --------------------------------------------------------------------------
# S5: cross-layer bonus
# --------------------------------------------------------------------------

def check_bonus_hand(adjusted_priority):
    """Hand-computed, exactly representable cases of P' = P + lambda*I*(1 - n/(l+1))."""
    p = np.array([[0.25, 0.5, 0.125, 0.0]], dtype=np.float32)
    imp = np.array([0.5, 0.25, 1.0, 0.75], dtype=np.float32)
    n = np.array([1, 0, 3, 2])
    keep = np.zeros((1, 4), dtype=bool)
    # layer 3 -> denominator 4: coverage = 1/4, 0, 3/4, 2/4
    got = adjusted_priority(p, imp, n, 3, 2.0, keep)
    want = np.array([[0.25 + 2 * 0.5 * 0.75, 0.5 + 2 * 0.25, 0.125 + 2 * 1.0 * 0.25,
                      0.0 + 2 * 0.75 * 0.5]], dtype=np.float32)
    np.testing.assert_array_equal(got, want)
    keep[0, 2] = True
    got = adjusted_priority(p, imp, n, 3, 2.0, keep)
    assert got[0, 2] == np.float32(1.0)
    # layer 0: nothing covered yet -> focus = I
    got0 = adjusted_priority(p, imp, np.zeros(4, int), 0, 1.0, np.zeros((1, 4), bool))
    np.testing.assert_array_equal(got0, (p + imp[None, :]).astype(np.float32))
    # lambda = 0 leaves P untouched
    got1 = adjusted_priority(p, imp, n, 3, 0.0, np.zeros((1, 4), bool))
    np.testing.assert_array_equal(got1, p)


def test_bonus_hand():
    check_bonus_hand(orc.adjusted_priority)


def test_bonus_fp32_single_rounding():
    """Each operation is one fp32 operation: compare with explicit fp32 steps
    computed through Python floats rounded after every operation."""
    r = _rng(17)
    p = r.random((2, 50)).astype(np.float32) * 1e-3
    imp = r.random(50).astype(np.float32) * 1e-2
    n = r.integers(0, 7, size=50)
    got = orc.adjusted_priority(p, imp, n, 6, 1.0, np.zeros((2, 50), bool))
    f = lambda v: float(np.float32(v))   # noqa: E731
    for h in range(2):
        for t in range(50):
            cov = f(f(n[t]) / f(7))
            want = f(f(p[h, t]) + f(f(1.0) * f(f(imp[t]) * f(1.0 - cov))))
            assert got[h, t] == np.float32(want)


# --------------------------------------------------------------------------
# whole layer on fp32 scores
# --------------------------------------------------------------------------

def _scores(seed, H, Tc, heavy=True):
    r = _rng(seed)
    p = (r.random((H, Tc)) ** 4 * 1e-3).astype(np.float32)
    pe = (p * (0.5 + r.random((H, Tc)))).astype(np.float32)
    imp = (p.max(axis=0) * (1 + r.random(Tc))).astype(np.float32)
    return p, pe, imp


def _sel(p, pe, imp, n_t, layer, **kw):
    return orc.select_layer(p, pe, imp, n_t, layer, **kw)


def test_layer_invariants():
    H, T, O, B = 4, 300, 8, 40
    p, pe, imp = _scores(18, H, T - O)
    n_t = _rng(19).integers(0, 3, size=T)
    res = _sel(p, pe, imp, n_t, 2, T=T, window=O, window_ext=16, budget=B, pool_kernel=5,
               delta=2, lam=1.0, beta=0.25)
    assert res.idx.shape == (H, B)
    for h in range(H):
        row = res.idx[h]
        assert len(set(row.tolist())) == B                    # exactly B distinct tokens
        assert list(row[B - O:]) == list(range(T - O, T))     # the window is kept
        pre = row[:B - O]
        assert np.all(np.diff(pre) > 0) and pre[-1] < T - O   # ascending prefix picks
        assert res.keep[h].sum() == orc.preserve_count(B, O, 0.25)
        assert set(np.nonzero(res.keep[h])[0].tolist()) <= set(pre.tolist())
    assert len(res.htop) == 2
    assert res.bits.sum() == len(set(res.idx.ravel().tolist()))


def test_reduces_to_snapkv_when_coverage_off():
    """delta = 0 and lambda = 0: plain top-(B-O) of the pooled window score, plus the window."""
    H, T, O, B = 3, 200, 6, 30
    p, pe, imp = _scores(20, H, T - O)
    n_t = _rng(21).integers(0, 4, size=T)
    res = _sel(p, pe, imp, n_t, 3, T=T, window=O, window_ext=12, budget=B, pool_kernel=7,
               delta=0, lam=0.0, beta=0.25)
    pooled = orc.maxpool1d(p, 7)
    for h in range(H):
        want = np.sort(orc.rank_first(pooled[h], B - O))
        np.testing.assert_array_equal(res.idx[h, :B - O], want)


def test_full_preserve_ignores_bonus():
    """beta*B >= B-O: every prefix pick is preserved, so the bonus cannot change the set."""
    H, T, O, B = 3, 150, 4, 20
    p, pe, imp = _scores(22, H, T - O)
    n_t = np.zeros(T, int)
    a = _sel(p, pe, imp, n_t, 0, T=T, window=O, window_ext=8, budget=B, pool_kernel=3,
             delta=1, lam=5.0, beta=1.0)
    b = _sel(p, pe, imp, n_t, 0, T=T, window=O, window_ext=8, budget=B, pool_kernel=3,
             delta=1, lam=0.0, beta=1.0)
    np.testing.assert_array_equal(a.idx, b.idx)


def check_preserve_uses_replaced_scores(select_layer):
    """Algorithm 1 replaces P by the extended-window score for H_top BEFORE picking the
    preserved tokens, so a head in H_top preserves its top tokens of P_ext."""
    T, O, B = 40, 2, 6          # 4 prefix picks, preserve 1 (beta = 0.25 -> floor(1.5) = 1)
    Tc = T - O
    p = np.full((2, Tc), 1e-3, np.float32)
    p[1, ::5] = 0.2             # head 1 is focused; head 0 (flat) has the lowest sigma
    p[0, 10] = 2e-3             # head 0's best token under P
    pe = p.copy()
    pe[0, 30] = 0.05            # head 0's best token under P_ext
    imp = np.zeros(Tc, np.float32)
    imp[12] = 0.9               # a big bonus elsewhere
    res = select_layer(p, pe, imp, np.zeros(T, int), 0, T=T, window=O, window_ext=4, budget=B,
                       pool_kernel=1, delta=1, lam=1.0, beta=0.25)
    assert list(res.htop) == [0]
    assert res.keep[0, 30] and not res.keep[0, 10]
    assert 30 in res.idx[0]


def test_preserve_uses_replaced_scores():
    check_preserve_uses_replaced_scores(orc.select_layer)


def test_preserve_beats_bonus():
    """A preserved token stays even when the coverage bonus lifts others above it."""
    T, O, B = 30, 2, 4          # 2 prefix picks, beta = 0.25 -> preserve 1
    Tc = T - O
    p = np.full((1, Tc), 1e-4, np.float32)
    p[0, 5] = 0.3
    imp = np.zeros(Tc, np.float32)
    imp[[9, 11]] = 0.8
    res = orc.select_layer(p, p, imp, np.zeros(T, int), 0, T=T, window=O, window_ext=O, budget=B,
                           pool_kernel=1, delta=0, lam=1.0, beta=0.25)
    assert list(res.idx[0, :2]) == [5, 9]       # without preservation: [9, 11]


def test_keep_everything_when_budget_covers_prefix():
    H, T, O, B = 2, 20, 4, 32
    p, pe, imp = _scores(23, H, T - O)
    res = _sel(p, pe, imp, np.zeros(T, int), 0, T=T, window=O, window_ext=8, budget=B,
               pool_kernel=3, delta=1, lam=1.0, beta=0.25)
    assert list(res.idx[0, :T]) == list(range(T))
    assert np.all(res.idx[:, T:] == -1)


def test_coverage_is_union_size():
    r = _rng(24)
    T = 100
    layers = []
    for _ in range(4):
        idx = np.stack([np.sort(r.choice(T, 10, replace=False)) for _ in range(3)]).astype(np.int32)
        layers.append(orc.layer_bits(idx, T))
    want = len(set().union(*[set(np.nonzero(b)[0].tolist()) for b in layers]))
    assert orc.coverage_count(layers) == want
    n_t = orc.counts_from_bits(layers[:3])
    assert n_t.max() <= 3


def check_counts_hand(counts_from_bits):
    """n_t (Sec. 4.2: the number of earlier layers that kept token t, the coverage
    counters of Algorithm 1), counted by hand over four known layer bitmaps."""
    rows = [np.array(r, dtype=bool) for r in (
        [1, 0, 1, 0, 1, 0, 0, 1, 0, 1],
        [1, 1, 0, 0, 1, 0, 0, 1, 0, 0],
        [0, 1, 0, 0, 1, 0, 1, 1, 0, 0],
        [1, 0, 0, 1, 1, 0, 0, 1, 0, 1])]
    # column totals written out by hand, not computed
    assert list(counts_from_bits(rows[:1])) == [1, 0, 1, 0, 1, 0, 0, 1, 0, 1]
    assert list(counts_from_bits(rows[:2])) == [2, 1, 1, 0, 2, 0, 0, 2, 0, 1]
    assert list(counts_from_bits(rows[:3])) == [2, 2, 1, 0, 3, 0, 1, 3, 0, 1]
    assert list(counts_from_bits(rows)) == [3, 2, 1, 1, 4, 0, 1, 4, 0, 2]


def test_counts_hand():
    check_counts_hand(orc.counts_from_bits)


def test_counts_from_kept_indices():
    """n_t from layer_bits of index sets: a token kept by two heads of one layer
    counts once for that layer; the window counts in every layer."""
    T = 12
    l0 = np.array([[0, 3, 10, 11], [3, 5, 10, 11]], dtype=np.int32)   # t = 3 kept by both heads
    l1 = np.array([[1, 3, 10, 11], [2, 7, 10, 11]], dtype=np.int32)
    n_t = orc.counts_from_bits([orc.layer_bits(l0, T), orc.layer_bits(l1, T)])
    assert list(n_t) == [1, 1, 1, 2, 0, 1, 0, 1, 0, 0, 2, 2]


def check_pool_before_sigma(select_layer):
    """Pooling comes before sigma, and the H_top heads take the POOLED P over O'.

    Head 0's raw P alternates 0.02 / 0: a large raw sigma, but max-pooling with
    kernel 3 makes it exactly flat (pooled sigma 0).  Head 1 is a smooth step
    (raw sigma 0.002).  With delta = 1, sigma of pooled P picks head 0; sigma of
    raw P would pick head 1.  Head 0's P over O' has one spike at t = 30 and a
    lower one at t = 5: pooled, the spike covers 29..31, so the three prefix picks
    are 29, 30, 31; unpooled they would be 30, 5 and then 0 (a tie at the floor).
    """
    T, O, B = 42, 2, 5                   # Tc = 40, three prefix picks, preserve floor(1.25) = 1
    Tc = T - O
    p = np.zeros((2, Tc), np.float32)
    p[0, ::2] = 0.02
    p[1, :20], p[1, 20:] = 0.001, 0.005
    pe = p.copy()
    pe[0] = 0.001
    pe[0, 30] = 0.5
    pe[0, 5] = 0.1
    imp = np.zeros(Tc, np.float32)
    res = select_layer(p, pe, imp, np.zeros(T, int), 1, T=T, window=O, window_ext=4, budget=B,
                       pool_kernel=3, delta=1, lam=0.0, beta=0.25)
    assert list(res.htop) == [0]
    assert list(res.idx[0, :3]) == [29, 30, 31]
    assert res.keep[0, 29] and res.keep[0].sum() == 1


def test_pool_before_sigma():
    check_pool_before_sigma(orc.select_layer)


def test_gather_rows():
    x = _rng(25).standard_normal((2, 10, 4))
    idx = np.array([[3, 1, 9, -1], [0, 0, 5, 2]], dtype=np.int32)
    g = orc.gather_rows(x, idx)
    np.testing.assert_array_equal(g[0, 0], x[0, 3])
    np.testing.assert_array_equal(g[1, 2], x[1, 5])
    assert np.all(g[0, 3] == 0)


# --------------------------------------------------------------------------
# mutation tests: a planted mistake in a copy of the oracle must fail a pin
# --------------------------------------------------------------------------

def _mut_no_causal(q_win, k, window, full=False):
    hq, wn, d = q_win.shape
    hkv, T, _ = k.shape
    g = hq // hkv
    abar = np.zeros((hkv, wn, T))
    for j in range(hq):
        s = (q_win[j] @ k[j // g].T) / math.sqrt(d)          # mistake: no causal mask
        e = np.exp(s - s.max(axis=1, keepdims=True))
        abar[j // g] += e / e.sum(axis=1, keepdims=True) / g
    O = window
    p = abar[:, wn - O:].sum(1) / O
    pe = abar.sum(1) / wn
    imp = abar[:, wn - O:].max(0).sum(0) / O
    tc = T if full else T - O
    return p[:, :tc], pe[:, :tc], imp[:tc]


def _mut_wrong_window(q_win, k, window, full=False):
    p, pe, imp = orc.window_scores(q_win, k, window, full)
    return pe, pe, imp                                       # mistake: P over O' rows


def _mut_query_head_max(q_win, k, window, full=False):
    hq, wn, d = q_win.shape
    hkv, T, _ = k.shape
    g = hq // hkv
    pos = T - wn + np.arange(wn)
    vis = np.arange(T)[None, :] <= pos[:, None]
    a = np.zeros((hq, wn, T))
    for j in range(hq):
        s = np.where(vis, (q_win[j] @ k[j // g].T) / math.sqrt(d), -np.inf)
        e = np.exp(s - s.max(1, keepdims=True))
        a[j] = e / e.sum(1, keepdims=True)
    abar = a.reshape(hkv, g, wn, T).mean(1)
    O = window
    p = abar[:, wn - O:].sum(1) / O
    pe = abar.sum(1) / wn
    imp = a[:, wn - O:].max(0).sum(0) / O                   # mistake: max over query heads
    tc = T if full else T - O
    return p[:, :tc], pe[:, :tc], imp[:tc]


def _mut_lse_no_causal(q_win, k):
    hq, wn, d = q_win.shape
    g = hq // k.shape[0]
    out = np.zeros((hq, wn))
    for j in range(hq):
        s = (q_win[j] @ k[j // g].T) / math.sqrt(d)          # mistake: every key visible
        m = s.max(axis=1)
        out[j] = m + np.log(np.exp(s - m[:, None]).sum(axis=1))
    return out


def _mut_lse_head_map(q_win, k):
    hq = q_win.shape[0]
    hkv = k.shape[0]
    out = np.zeros(q_win.shape[:2])
    for j in range(hq):                                       # mistake: j % H_kv, not j // G
        out[j] = orc.window_lse(q_win[j:j + 1], k[j % hkv:j % hkv + 1])[0]
    return out


def _mut_lse_no_scale(q_win, k):
    d = q_win.shape[2]
    return orc.window_lse(q_win * math.sqrt(d), k)            # mistake: scale 1/sqrt(d) dropped


def _mut_entropy_unnormalised(p):
    x = np.asarray(p, dtype=np.float64)
    out = np.zeros(x.shape[0])
    for h in range(x.shape[0]):
        q = x[h][x[h] > 0]                                    # mistake: not divided by the sum
        out[h] = -(q * np.log(q)).sum()
    return out


def _mut_entropy_lowest(pooled, delta, criterion="std"):
    if criterion == "entropy":
        return orc.adjusted_heads(orc.head_entropy(pooled), delta)   # mistake: most focused
    return orc.focus_heads(pooled, delta, criterion)


def _mut_decode_head_map(q, k, v, valid=None):
    hq, hkv = q.shape[0], k.shape[0]
    out = np.zeros(q.shape)
    for j in range(hq):                                       # mistake: j % H_kv, not j // G
        out[j] = orc.decode_attention(q[j:j + 1], k[j % hkv:j % hkv + 1], v[j % hkv:j % hkv + 1],
                                      None if valid is None else valid[j % hkv:j % hkv + 1])[0]
    return out


def _mut_decode_no_scale(q, k, v, valid=None):
    return orc.decode_attention(q * math.sqrt(q.shape[1]), k, v, valid)   # mistake: no 1/sqrt(d)


def _mut_decode_no_mask(q, k, v, valid=None):
    return orc.decode_attention(q, k, v, None)                           # mistake: mask ignored


def _mut_highest_sigma(sigma, delta):
    order = sorted(range(len(sigma)), key=lambda h: (-float(sigma[h]), h))   # mistake
    return np.array(sorted(order[:delta]), dtype=np.int64)


def _mut_layer_denominator(p_sel, imp, n_t, layer, lam, keep):
    f32 = np.float32
    cov = n_t.astype(f32) / f32(max(layer, 1))               # mistake: l instead of l+1
    out = p_sel.astype(f32) + f32(lam) * (imp.astype(f32) * (f32(1) - cov))[None, :]
    out[keep] = f32(1)
    return out


def _mut_sample_std(p):
    x = np.asarray(p, dtype=np.float64)
    return x.std(axis=1, ddof=1)                              # mistake: sample std


def _mut_rank_index_desc(scores, k):
    n = scores.shape[0]
    return np.lexsort((-np.arange(n), -np.asarray(scores, np.float64)))[:k]   # mistake: ties


def _mut_maxpool_shift(x, kernel):
    out = orc.maxpool1d(x, kernel)
    return np.concatenate([out[..., 1:], out[..., -1:]], axis=-1)            # mistake: off by one


def _mut_preserve_raw(p_raw, p_ext_raw, imp, n_t, layer, **kw):
    """Mistake: preserve set taken from P before the H_top replacement."""
    res = orc.select_layer(p_raw, p_ext_raw, imp, n_t, layer, **kw)
    H, Tc = p_raw.shape
    pooled = orc.maxpool1d(p_raw.astype(np.float32), kw["pool_kernel"])
    kp = orc.preserve_count(kw["budget"], kw["window"], kw["beta"])
    keep = np.zeros((H, Tc), bool)
    for h in range(H):
        keep[h, orc.rank_first(pooled[h], kp)] = True
    res.keep = keep
    padj = orc.adjusted_priority(res.p_sel, imp, np.asarray(n_t)[:Tc], layer, kw["lam"], keep)
    m = kw["budget"] - kw["window"]
    for h in range(H):
        res.idx[h, :m] = np.sort(orc.rank_first(padj[h], m))
    return res


def _mut_counts_or(layer_bits_list):
    """Mistake: a token kept in any earlier layer counts once (OR instead of a sum)."""
    u = np.zeros_like(np.asarray(layer_bits_list[0], dtype=bool))
    for b in layer_bits_list:
        u |= np.asarray(b, dtype=bool)
    return u.astype(np.int64)


def _mut_counts_last(layer_bits_list):
    """Mistake: only the previous layer is counted."""
    return np.asarray(layer_bits_list[-1], dtype=np.int64)


def _select_variant(p_raw, p_ext_raw, imp, n_t, layer, *, sigma_raw=False, ext_unpooled=False,
                    T, window, window_ext, budget, pool_kernel, delta, lam, beta):
    """select_layer with one of two planted mistakes in the order of operations."""
    O = window
    Tc = T - O
    H = p_raw.shape[0]
    pooled = orc.maxpool1d(p_raw.astype(np.float32), pool_kernel)
    pooled_ext = orc.maxpool1d(p_ext_raw.astype(np.float32), pool_kernel)
    sig = orc.head_sigma(p_raw if sigma_raw else pooled)
    htop = orc.adjusted_heads(sig, delta) if min(window_ext, T) > O else np.zeros(0, np.int64)
    p_sel = pooled.copy()
    p_sel[htop] = (p_ext_raw if ext_unpooled else pooled_ext)[htop]
    kp = orc.preserve_count(budget, O, beta)
    keep = np.zeros((H, Tc), dtype=bool)
    for h in range(H):
        keep[h, orc.rank_first(p_sel[h], kp)] = True
    p_adj = orc.adjusted_priority(p_sel, imp, np.asarray(n_t)[:Tc], layer, lam, keep)
    m = budget - O
    idx = np.empty((H, budget), dtype=np.int32)
    for h in range(H):
        idx[h, :m] = np.sort(orc.rank_first(p_adj[h], m))
        idx[h, m:] = np.arange(Tc, T)
    return orc.LayerResult(idx, htop, sig, keep, p_sel, p_adj, np.zeros(T, bool))


def _mut_sigma_raw(*a, **kw):
    return _select_variant(*a, sigma_raw=True, **kw)


def _mut_ext_unpooled(*a, **kw):
    return _select_variant(*a, ext_unpooled=True, **kw)


def test_select_variant_matches_oracle_without_mistakes():
    """The mutation harness itself reproduces the oracle when no mistake is planted."""
    H, T, O, B = 4, 300, 8, 40
    p, pe, imp = _scores(31, H, T - O)
    n_t = _rng(32).integers(0, 3, size=T)
    kw = dict(T=T, window=O, window_ext=16, budget=B, pool_kernel=5, delta=2, lam=1.0, beta=0.25)
    a = orc.select_layer(p, pe, imp, n_t, 3, **kw)
    b = _select_variant(p, pe, imp, n_t, 3, **kw)
    np.testing.assert_array_equal(a.idx, b.idx)
    np.testing.assert_array_equal(a.htop, b.htop)


@pytest.mark.parametrize("check,mutant", [
    (check_zero_query_closed_form, _mut_no_causal),
    (check_zero_query_closed_form, _mut_wrong_window),
    (check_brute_force, _mut_no_causal),
    (check_brute_force, _mut_query_head_max),
    (check_lse_constant_keys, _mut_lse_no_causal),
    (check_lse_constant_keys, _mut_lse_head_map),
    (check_lse_constant_keys, _mut_lse_no_scale),
    (check_lse_brute, _mut_lse_no_causal),
    (check_lse_normalises_scores, _mut_lse_no_scale),
    (check_lowest_sigma, _mut_highest_sigma),
    (check_decode_constant_keys, _mut_decode_head_map),
    (check_decode_constant_keys, _mut_decode_no_mask),
    (check_decode_brute, _mut_decode_no_scale),
    (check_decode_brute, _mut_decode_head_map),
    (check_entropy_closed_forms, _mut_entropy_unnormalised),
    (check_entropy_brute, _mut_entropy_unnormalised),
    (check_entropy_picks_least_focused, _mut_entropy_lowest),
    (check_bonus_hand, _mut_layer_denominator),
    (check_sigma, _mut_sample_std),
    (check_rank_brute, _mut_rank_index_desc),
    (check_maxpool, _mut_maxpool_shift),
    (check_preserve_uses_replaced_scores, _mut_preserve_raw),
    (check_counts_hand, _mut_counts_or),
    (check_counts_hand, _mut_counts_last),
    (check_pool_before_sigma, _mut_sigma_raw),
    (check_pool_before_sigma, _mut_ext_unpooled),
])
def test_pins_catch_planted_mistakes(check, mutant):
    with pytest.raises(AssertionError):
        check(mutant)
