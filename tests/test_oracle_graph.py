"""Pins of the oracle boosting graph against things other than itself.

* graph states: brute-force longest-suffix enumeration over whole hypotheses
  (the oracle advances incrementally with the Aho-Corasick move);
* potentials: hand-derived worked examples (tests/golden/, Sec. II-A);
* pure-potential reading: its closed form for the summed step boosts;
* commit reading: a lone phrase earns w per token plus the end bonus, a broken
  match loses exactly its pending part;
* case insensitivity (Sec. II-A): case variants give the same graph.
"""

import itertools
import os

import numpy as np
import pytest

import oracle
from oracle.graph import COMMIT, PURE_POTENTIAL, build_graph
from tests import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _identity_cm(n):
    cm = np.arange(n + 1, dtype=np.int32)
    cm[n] = -1
    return cm


def _walk(g, h):
    s = 0
    out = []
    for c in h:
        s = g.delta(s, c)
        out.append(s)
    return out


@pytest.mark.parametrize("seed", range(12))
def test_states_match_brute_force(seed):
    rng = np.random.default_rng(seed)
    n_sym = 4
    F = [tuple(rng.integers(0, n_sym, size=rng.integers(1, 5))) for _ in range(rng.integers(1, 7))]
    g = build_graph([list(f) for f in F], _identity_cm(n_sym + 1))
    pref = brute.prefixes(F)
    assert sorted(g.strings, key=lambda x: (len(x), x)) == sorted(pref, key=lambda x: (len(x), x))
    for h in brute.all_strings(n_sym + 1, 6):  # includes a symbol in no phrase
        sts = _walk(g, h)
        for t in range(len(h)):
            assert g.strings[sts[t]] == brute.sigma(h[:t + 1], pref)
    # suffix links: longest proper suffix in Pref
    for sid, x in enumerate(g.strings):
        if sid:
            assert g.strings[g.link[sid]] == brute.sigma(x[1:], pref)


def test_breadth_first_numbering():
    g = build_graph([[2, 0], [0, 1], [1], [0, 0, 3]], _identity_cm(5))
    depth_then_parent = [(len(x), g.strings.index(x[:-1]) if x else -1, x[-1] if x else -1)
                         for x in g.strings]
    assert depth_then_parent == sorted(depth_then_parent)
    assert g.strings[0] == ()


@pytest.mark.parametrize("fname,sem", [("worked_example_commit.txt", COMMIT),
                                       ("worked_example_pure.txt", PURE_POTENTIAL)])
def test_worked_example(fname, sem):
    phrases, w, B, states, hyps = brute.parse_golden(os.path.join(GOLDEN, fname))
    g = build_graph([list(p) for p in phrases], _identity_cm(5), token_w=w, end_bonus=B,
                    semantics=sem)
    assert g.n_states == len(states)
    for sid, string, link, phi, E, psi in states:
        assert g.strings[sid] == string
        assert g.link[sid] == link
        assert g.phi64[sid] == phi and g.e64[sid] == E and g.psi64[sid] == psi
    for toks, boosts, sts in hyps:
        s = 0
        for t, c in enumerate(toks):
            ns = g.delta(s, c)
            assert ns == sts[t]
            assert g.phi64[ns] - g.phi64[s] + g.e64[ns] == boosts[t]
            s = ns


@pytest.mark.parametrize("seed", range(8))
def test_pure_potential_closed_form(seed):
    """Sum of step boosts = a*w*|sigma(h)| + a*B * #{t: a suffix of sigma(h_<=t) is a phrase}."""
    rng = np.random.default_rng(100 + seed)
    n_sym, w, B, a = 4, 0.75, 1.5, 1.25
    F = [tuple(rng.integers(0, n_sym, size=rng.integers(1, 5))) for _ in range(5)]
    g = build_graph([list(f) for f in F], _identity_cm(n_sym + 1), token_w=w, end_bonus=B,
                    alpha=a, semantics=PURE_POTENTIAL)
    pref, Fs = brute.prefixes(F), set(F)
    for _ in range(200):
        h = tuple(rng.integers(0, n_sym + 1, size=rng.integers(0, 9)))
        s, tot, arrivals = 0, 0.0, 0
        for t, c in enumerate(h):
            ns = g.delta(s, c)
            tot += g.psi64[ns] - g.phi64[s]
            s = ns
            sig = brute.sigma(h[:t + 1], pref)
            arrivals += any(sig[i:] in Fs for i in range(len(sig)))
        expect = a * w * len(brute.sigma(h, pref)) + a * B * arrivals
        assert abs(tot - expect) < 1e-12


def test_commit_lone_phrase_and_cancellation():
    """A phrase spelled alone earns w per token plus B; a broken match pays back its pending part."""
    w, B = 1.5, 2.5
    F = [(0, 1, 2, 3), (4, 5)]
    g = build_graph([list(f) for f in F], _identity_cm(7), token_w=w, end_bonus=B)
    for f in F:
        s, tot, partial = 0, 0.0, []
        for c in f:
            ns = g.delta(s, c)
            tot += g.phi64[ns] - g.phi64[s] + g.e64[ns]
            partial.append(tot)
            s = ns
        assert tot == w * len(f) + B
        assert partial[:-1] == [w * (i + 1) for i in range(len(f) - 1)]
    # break after every partial prefix with symbol 6 (in no phrase): total returns to 0
    for L in range(1, 4):
        s, tot = 0, 0.0
        for c in F[0][:L] + (6,):
            ns = g.delta(s, c)
            tot += g.phi64[ns] - g.phi64[s] + g.e64[ns]
            s = ns
        assert s == 0 and tot == 0.0


def test_case_variants_give_same_graph():
    """Sec. II-A: a phrase written in any case variant is the same graph."""
    from workloads import Config, class_map
    cfg = Config(0, "t", B=1, K=1, V=30, T=1, chunk=1, dtype="f32", n_phrases=0, len_lo=1,
                 len_hi=1, token_dist="uniform", zipf_s=0, logit_std=1, blank_offset=0, n_case=8)
    cm = class_map(cfg)
    base = [[1, 2, 3], [2, 20], [5]]
    rng = np.random.default_rng(0)
    g0 = build_graph(base, cm)
    for _ in range(10):
        var = [[int(t + 8 * rng.integers(0, 3)) if t < 8 else t for t in p] for p in base]
        g1 = build_graph(var, cm)
        assert g1.strings == g0.strings and g1.link == g0.link
        assert np.array_equal(g1.psi32, g0.psi32) and np.array_equal(g1.phi32, g0.phi32)
    # every case variant of a token moves to the same state
    for s in range(g0.n_states):
        row = g0.token_row(s)
        for t in range(8):
            assert row[t] == row[t + 8] == row[t + 16]


def test_empty_and_duplicate_lists():
    cm = _identity_cm(4)
    g = build_graph([], cm)
    assert g.n_states == 1 and g.psi64[0] == 0 and g.phi64[0] == 0
    assert np.all(g.token_row(0) == 0)
    g1 = build_graph([[1, 2], [1, 2], [1]], cm)
    g2 = build_graph([[1], [1, 2]], cm)
    assert g1.strings == g2.strings and np.array_equal(g1.psi64, g2.psi64)


def test_rejects_bad_phrases():
    cm = _identity_cm(4)
    with pytest.raises(ValueError):
        build_graph([[]], cm)
    with pytest.raises(ValueError):
        build_graph([[4]], cm)   # the blank
    with pytest.raises(ValueError):
        build_graph([[7]], cm)
