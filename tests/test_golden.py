"""Both oracles against the hand-derived fixtures of tests/golden/ (each file
names the passage it follows and gives its derivation)."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle as orc
from oracle import cxx

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
ORACLES = [("numpy", orc), ("cxx", cxx)]


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _num(v):
    return float(Fraction(v)) if isinstance(v, str) else float(v)


@pytest.fixture(scope="module", autouse=True)
def _built():
    cxx.build(force=False)


@pytest.mark.parametrize("name,o", ORACLES, ids=[n for n, _ in ORACLES])
def test_window_scores_zero_query(name, o):
    g = _load("window_scores_zero_query.json")
    s = g["shape"]
    q = np.zeros((s["hq"], s["window_rows"], s["d"]))
    k = np.random.default_rng(0).standard_normal((s["hkv"], s["T"], s["d"]))
    p, pe, imp = o.window_scores(q, k, s["O"])
    for h in range(s["hkv"]):
        np.testing.assert_allclose(p[h], [_num(x) for x in g["P"]], rtol=1e-14)
        np.testing.assert_allclose(pe[h], [_num(x) for x in g["P_ext"]], rtol=1e-14)
    np.testing.assert_allclose(imp, [_num(x) for x in g["I"]], rtol=1e-14)


@pytest.mark.parametrize("name,o", ORACLES, ids=[n for n, _ in ORACLES])
def test_coverage_counts(name, o):
    g = _load("coverage_counts.json")
    rows = [np.array(r, dtype=bool) for r in g["rows"]]
    for k, want in enumerate(g["counts_after"], start=1):
        assert list(o.counts_from_bits(rows[:k])) == want
    assert o.coverage_count(rows) == g["coverage"]


@pytest.mark.parametrize("name,o", ORACLES, ids=[n for n, _ in ORACLES])
def test_coverage_bonus(name, o):
    g = _load("coverage_bonus.json")
    p = np.array([g["p"]], dtype=np.float32)
    imp = np.array(g["imp"], dtype=np.float32)
    n = np.array(g["n"])
    got = o.adjusted_priority(p, imp, n, g["layer"], g["lam"], np.zeros((1, len(n)), bool))
    np.testing.assert_array_equal(got[0], np.array(g["expected"], dtype=np.float32))
    got = o.adjusted_priority(p, imp, n, g["layer"], g["lam"], np.array([g["preserved"]]))
    np.testing.assert_array_equal(got[0], np.array(g["expected_preserved"], dtype=np.float32))


@pytest.mark.parametrize("name,o", ORACLES, ids=[n for n, _ in ORACLES])
def test_preserve_count(name, o):
    for B, O, beta, want in _load("preserve_count.json")["cases"]:
        assert o.preserve_count(B, O, beta) == want, (B, O, beta)


@pytest.mark.parametrize("name,o", ORACLES, ids=[n for n, _ in ORACLES])
def test_rank_ties(name, o):
    g = _load("rank_ties.json")
    s = np.array(g["scores"], dtype=np.float32)
    for k in range(len(s) + 1):
        assert list(o.rank_first(s, k)) == g["order"][:k]
