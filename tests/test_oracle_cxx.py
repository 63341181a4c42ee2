"""The C++ oracle (oracle/kvec_oracle.cpp) against the same pins as the numpy
oracle, and the two oracles against each other.

The pins are the closed forms, brute force and hand-computed cases of
test_oracle_pins.py, applied unchanged to the C++ routines; the cross-checks
run both oracles on random inputs of several shapes and policies (float64
scores within a few ulps, the fp32 policy results bit-exact).  Nothing here
calls the GPU.
"""
import numpy as np
import pytest

import oracle as orc
import synth
import test_oracle_pins as pins
from oracle import cxx


@pytest.fixture(scope="module", autouse=True)
def _built():
    cxx.build(force=False)


# --- the pins, on the C++ routines -----------------------------------------

@pytest.mark.parametrize("check", [
    pins.check_zero_query_closed_form, pins.check_brute_force, pins.check_mass,
    pins.check_identical_heads, pins.check_single_row_softmax])
def test_window_score_pins(check):
    check(cxx.window_scores)


@pytest.mark.parametrize("check", [
    pins.check_lse_constant_keys, pins.check_lse_brute, pins.check_lse_normalises_scores])
def test_lse_pins(check):
    check(cxx.window_lse)


@pytest.mark.parametrize("check", [pins.check_decode_constant_keys, pins.check_decode_brute])
def test_decode_pins(check):
    check(cxx.decode_attention)


def test_selection_pins():
    pins.check_maxpool(cxx.maxpool1d)
    pins.check_sigma(cxx.head_sigma)
    pins.check_lowest_sigma(cxx.adjusted_heads)
    pins.check_entropy_closed_forms(cxx.head_entropy)
    pins.check_entropy_brute(cxx.head_entropy)
    pins.check_entropy_picks_least_focused(cxx.focus_heads)
    pins.check_rank_brute(cxx.rank_first)
    pins.check_bonus_hand(cxx.adjusted_priority)
    pins.check_preserve_uses_replaced_scores(cxx.select_layer)
    pins.check_counts_hand(cxx.counts_from_bits)
    pins.check_pool_before_sigma(cxx.select_layer)


def test_preserve_count_and_coverage():
    for B, O, beta in [(128, 32, 0.25), (1024, 32, 0.25), (40, 8, 1.0), (40, 8, 0.0), (10, 2, 0.33)]:
        assert cxx.preserve_count(B, O, beta) == orc.preserve_count(B, O, beta)
    bits = [np.array([1, 0, 0, 1, 0], bool), np.array([0, 0, 1, 1, 0], bool)]
    assert cxx.coverage_count(bits) == 3
    x = np.arange(2 * 10 * 4, dtype=np.float64).reshape(2, 10, 4)
    idx = np.array([[3, 1, 9, -1], [0, 0, 5, 2]], dtype=np.int32)
    np.testing.assert_array_equal(cxx.gather_rows(x, idx), orc.gather_rows(x, idx))


# --- the two oracles against each other ------------------------------------

@pytest.mark.parametrize("hq,hkv,wn,O,T,d", [
    (8, 4, 16, 8, 200, 32), (4, 4, 8, 8, 64, 16), (14, 2, 12, 4, 150, 8), (8, 1, 6, 3, 40, 64)])
def test_scores_match_numpy_oracle(hq, hkv, wn, O, T, d):
    r = np.random.default_rng(hq * 1000 + T)
    q = r.standard_normal((hq, wn, d))
    k = r.standard_normal((hkv, T, d)) * 1.5
    for full in (False, True):
        a = orc.window_scores(q, k, O, full=full)
        b = cxx.window_scores(q, k, O, full=full)
        for x, y in zip(a, b):
            np.testing.assert_allclose(y, x, rtol=1e-12, atol=0)
    np.testing.assert_allclose(cxx.window_lse(q, k), orc.window_lse(q, k), rtol=1e-13, atol=1e-13)
    # threads do not change the result
    np.testing.assert_array_equal(cxx.window_scores(q, k, O, threads=1)[0],
                                  cxx.window_scores(q, k, O, threads=5)[0])


def test_decode_matches_numpy_oracle():
    r = np.random.default_rng(5)
    q = r.standard_normal((8, 32))
    k = r.standard_normal((2, 50, 32))
    v = r.standard_normal((2, 50, 32))
    valid = r.random((2, 50)) < 0.7
    valid[1] = False
    for vm in (None, valid):
        np.testing.assert_allclose(cxx.decode_attention(q, k, v, vm), orc.decode_attention(q, k, v, vm),
                                   rtol=1e-12, atol=1e-14)


POLICIES = [
    dict(pool_kernel=7, delta=3, lam=1.0, beta=0.25),
    dict(pool_kernel=5, delta=2, lam=0.5, beta=0.5),
    dict(pool_kernel=1, delta=0, lam=0.0, beta=0.25),
    dict(pool_kernel=3, delta=4, lam=1.0, beta=1.0),
    dict(pool_kernel=7, delta=1, lam=2.0, beta=0.0, criterion="entropy"),
]


@pytest.mark.parametrize("pol", range(len(POLICIES)))
@pytest.mark.parametrize("layer", [0, 3])
def test_select_layer_matches_numpy_oracle(pol, layer):
    kw = POLICIES[pol]
    H, T, O, Oe, B = 4, 400, 8, 16, 48
    r = np.random.default_rng(pol * 10 + layer)
    p = (r.random((H, T - O)) ** 4 * 1e-3).astype(np.float32)
    p[:, ::37] = p[:, 1::37]                      # exact ties
    pe = (p * (0.5 + r.random((H, T - O)))).astype(np.float32)
    imp = (p.max(axis=0) * (1 + r.random(T - O))).astype(np.float32)
    n_t = r.integers(0, layer + 1, size=T)
    a = orc.select_layer(p, pe, imp, n_t, layer, T=T, window=O, window_ext=Oe, budget=B, **kw)
    b = cxx.select_layer(p, pe, imp, n_t, layer, T=T, window=O, window_ext=Oe, budget=B, **kw)
    np.testing.assert_array_equal(b.idx, a.idx)
    np.testing.assert_array_equal(b.htop, a.htop)
    np.testing.assert_array_equal(b.keep, a.keep)
    np.testing.assert_array_equal(b.p_sel.view(np.uint32), a.p_sel.view(np.uint32))
    np.testing.assert_array_equal(b.p_adj.view(np.uint32), a.p_adj.view(np.uint32))
    np.testing.assert_array_equal(b.bits, a.bits)
    np.testing.assert_allclose(b.sigma, a.sigma, rtol=1e-12)


def test_keep_everything_case_matches():
    H, T, O, B = 2, 20, 4, 32
    p = np.ones((H, T - O), np.float32)
    a = orc.select_layer(p, p, p[0], np.zeros(T, int), 0, T=T, window=O, window_ext=8, budget=B,
                         pool_kernel=3, delta=1, lam=1.0, beta=0.25)
    b = cxx.select_layer(p, p, p[0], np.zeros(T, int), 0, T=T, window=O, window_ext=8, budget=B,
                         pool_kernel=3, delta=1, lam=1.0, beta=0.25)
    np.testing.assert_array_equal(b.idx, a.idx)
    np.testing.assert_array_equal(b.bits, a.bits)


def test_tiny_workload_step_matches_numpy_oracle():
    """The tiny fp32 workload, every layer in order (n_t from the earlier
    layers' kept sets): both oracles keep the same tokens."""
    w = synth.workload(0)
    prev_a, prev_b = [], []
    for l in range(w.n_layers):
        q = synth.to_f64(synth.queries(w, l, 0), w.dtype)
        k = synth.to_f64(synth.keys(w, l, 0), w.dtype)
        sa = orc.score_layer(q, k, w.window)
        sb = cxx.score_layer(q, k, w.window)
        for x, y in zip(sa, sb):
            # fp32 scores: at most one rounding step apart
            assert np.max(np.abs(x.view(np.int32).astype(np.int64) - y.view(np.int32).astype(np.int64))) <= 1
        nta = orc.counts_from_bits(prev_a) if prev_a else np.zeros(w.seq_len, np.int64)
        ntb = cxx.counts_from_bits(prev_b) if prev_b else np.zeros(w.seq_len, np.int64)
        np.testing.assert_array_equal(ntb, nta)
        ra = orc.evict_layer_from_scores(*sa, nta, l, w)
        rb = cxx.evict_layer_from_scores(*sa, ntb, l, w)   # same fp32 scores: same picks
        np.testing.assert_array_equal(rb.idx, ra.idx)
        prev_a.append(ra.bits)
        prev_b.append(rb.bits)
    assert cxx.coverage_count(prev_b) == orc.coverage_count(prev_a)
