"""Pins of the oracle's variative BPE graph (Sec. II-A, Fig. 1c/1e, Eq. (1)).

* Eq. (1): tau = 0 splits a token's score evenly; the shares of one token add
  up to its score; a large tau puts nearly all of it on the last character,
  and consecutive shares at tau = 1 grow by the factor e;
* a vocabulary of single characters only reduces the variative graph to the
  class graph over characters (the already pinned oracle graph): same states,
  links, moves and potentials;
* every segmentation of a phrase into pieces, in every available casing, is
  accepted from the root and earns the same total boost, the phrase's score
  plus its end bonus (the paper: every accepted spelling receives the same
  total phrase bonus, independent of its BPE segmentation);
* the moves of the Aho-Corasick construction equal the moves defined from
  the strings alone (longest suffix node that can take the piece);
* the arc encoding: children contiguous with ascending classes, every arc's
  node is its source node extended by its piece, links are the longest proper
  suffix nodes, each node's first arc has the smallest id among its arcs;
* case invariance: cased phrases give the same graph.
"""

import math
import random

import numpy as np
import pytest

import oracle
from oracle.graph import COMMIT, PURE_POTENTIAL
from oracle.variative import build_variative_graph, eq1_split, move_by_strings

# characters: 0..25 lowercase letters, 26 = word start, 27..52 uppercase letters
LOWER = np.array(list(range(27)) + list(range(26)), dtype=np.int32)


def _s(text):
    out = []
    for ch in text:
        if ch == "_":
            out.append(26)
        elif ch.islower():
            out.append(ord(ch) - 97)
        else:
            out.append(27 + ord(ch) - 65)
    return tuple(out)


def _vocab(extra):
    """Single characters (lower, '_', upper) followed by the given pieces."""
    chars = [(c,) for c in range(53)]
    return chars + [_s(t) for t in extra]


@pytest.mark.parametrize("m", [1, 2, 3, 7])
def test_eq1_tau_zero_is_uniform(m):
    d = eq1_split(3.0, m, 0.0)
    assert all(abs(x - 3.0 / m) < 1e-15 for x in d)


@pytest.mark.parametrize("tau", [0.0, 0.5, 1.0, 2.0])
@pytest.mark.parametrize("m", [1, 2, 4, 6])
def test_eq1_shares_add_up_to_the_score(tau, m):
    assert abs(math.fsum(eq1_split(1.7, m, tau)) - 1.7) < 1e-14
    if tau > 0 and m > 1:
        d = eq1_split(1.7, m, tau)
        assert all(d[i] < d[i + 1] for i in range(m - 1))   # concentrated near the end


def test_eq1_large_tau_concentrates_on_the_last_character():
    d = eq1_split(1.0, 4, 3.0)
    assert d[-1] > 1.0 - 1e-15 and sum(d[:-1]) < 1e-15


def test_eq1_tau_one_ratio_is_e():
    d = eq1_split(1.0, 5, 1.0)
    for i in range(4):
        assert abs(d[i + 1] / d[i] - math.e) < 1e-12


@pytest.mark.parametrize("semantics", [COMMIT, PURE_POTENTIAL])
@pytest.mark.parametrize("seed", range(4))
def test_single_character_vocabulary_reduces_to_the_class_graph(semantics, seed):
    rng = random.Random(seed)
    words = ["".join(rng.choice("abcde_") for _ in range(rng.randint(1, 6))) for _ in range(12)]
    vocab = _vocab([])
    phrases = [_s(w) for w in words]
    g = build_variative_graph(vocab, LOWER, phrases, token_w=1.25, end_bonus=2.0, alpha=0.8,
                              tau=rng.choice([0.0, 1.0, 2.5]), semantics=semantics)
    cm = oracle.class_map_of(vocab, LOWER)
    ref = oracle.build_graph(phrases, cm, token_w=1.25, end_bonus=2.0, alpha=0.8,
                             semantics=semantics)
    assert g.n_states == ref.n_states
    assert [tuple(int(cm[c]) for c in s) for s in g.strings] == ref.strings
    assert g.goto == ref.goto and g.link == ref.link
    assert np.array_equal(g.phi32, ref.phi32) and np.array_equal(g.psi32, ref.psi32)
    for s in range(g.n_states):
        assert np.array_equal(g.token_row(s), ref.token_row(s))


def _segmentations(p, pieces):
    if not p:
        yield []
        return
    for m in range(1, len(p) + 1):
        if p[:m] in pieces:
            for rest in _segmentations(p[m:], pieces):
                yield [p[:m]] + rest


@pytest.mark.parametrize("tau", [0.0, 1.0, 2.0])
@pytest.mark.parametrize("word", ["_hello", "_help_me", "_aaa", "_abcab"])
def test_every_segmentation_and_casing_earns_the_same_total(tau, word):
    extra = ["_he", "_He", "_HE", "ll", "LL", "hel", "el", "lo", "_help", "_Help", "me", "_me",
             "aa", "AA", "_a", "ab", "Ab", "bca", "cab", "_ab"]
    vocab = _vocab(extra)
    cm = oracle.class_map_of(vocab, LOWER)
    can = oracle.variative.canon_strings(vocab, LOWER)
    by_canon = {}
    for v, c in enumerate(can):
        by_canon.setdefault(c, []).append(v)
    p = _s(word)
    g = build_variative_graph(vocab, LOWER, [p], token_w=1.5, end_bonus=2.0, alpha=1.0, tau=tau)
    n_backbone = len(oracle.variative.greedy_backbone(p, set(can)))
    want = 1.0 * (1.5 * n_backbone + 2.0)
    segs = list(_segmentations(p, set(can)))
    assert len(segs) >= 2
    rng = random.Random(7)
    for seg in segs:
        for _ in range(3):
            s, total = 0, 0.0
            for piece in seg:
                v = rng.choice(by_canon[piece])          # any casing of the piece
                d = int(g.token_row(s)[v])
                total += float(g.psi64[d]) - float(g.phi64[s])
                s = d
            assert g.strings[s] == p
            assert abs(total - want) < 1e-12, (seg, total, want)


@pytest.mark.parametrize("seed", range(5))
def test_moves_equal_the_string_definition(seed):
    rng = random.Random(100 + seed)
    letters = "abc_"
    extra = list({"".join(rng.choice(letters) for _ in range(rng.randint(2, 4))) for _ in range(14)})
    extra += [e.upper() for e in extra[:4] if e.upper() != e]
    vocab = _vocab(extra)
    phrases = [_s("".join(rng.choice(letters) for _ in range(rng.randint(1, 7)))) for _ in range(8)]
    g = build_variative_graph(vocab, LOWER, phrases, tau=1.0)
    for s in range(g.n_states):
        row = g.token_row(s)
        for v in range(len(vocab)):
            assert row[v] == move_by_strings(g, vocab, LOWER, s, v), (s, v)


@pytest.mark.parametrize("seed", range(5))
def test_arc_encoding(seed):
    rng = random.Random(200 + seed)
    letters = "abcd_"
    extra = list({"".join(rng.choice(letters) for _ in range(rng.randint(2, 5))) for _ in range(20)})
    vocab = _vocab(extra)
    can = oracle.variative.canon_strings(vocab, LOWER)
    cm = oracle.class_map_of(vocab, LOWER)
    cstr = {int(cm[v]): can[v] for v in range(len(vocab))}
    phrases = [_s("".join(rng.choice(letters) for _ in range(rng.randint(1, 8)))) for _ in range(10)]
    g = build_variative_graph(vocab, LOWER, phrases, tau=0.5)
    nodes = set(g.strings)
    first = {}
    for sid, T in enumerate(g.strings):
        first.setdefault(T, sid)
        kids = sorted(g.goto[sid].items())
        ids = [y for _, y in kids]
        assert ids == list(range(ids[0], ids[0] + len(ids))) if ids else True
        for c, y in kids:
            assert g.strings[y] == T + cstr[c]
            assert all(g.goto[x] == g.goto[sid] for x in range(g.n_states) if g.strings[x] == T)
        # link: first arc into the longest proper suffix node
        suf = next((T[i:] for i in range(1, len(T) + 1) if T[i:] in nodes), ())
        assert g.link[sid] == (min(x for x in range(g.n_states) if g.strings[x] == suf)
                               if T else 0)
    # every node is reached, and its first arc has the smallest id of its arcs
    assert set(first) == nodes
    for T, f in first.items():
        assert all(f <= x for x in range(g.n_states) if g.strings[x] == T)
    # nodes expanded by length: the child blocks appear in order of node length
    order = sorted(set((min(g.goto[s].values()), len(g.strings[s])) for s in range(g.n_states)
                       if g.goto[s]))
    assert [L for _, L in order] == sorted(L for _, L in order)


def test_cased_phrases_give_the_same_graph():
    vocab = _vocab(["_he", "_He", "llo", "LLO", "_wor", "ld"])
    a = build_variative_graph(vocab, LOWER, [_s("_hello"), _s("_world")], tau=1.0)
    b = build_variative_graph(vocab, LOWER, [_s("_HeLLo"), _s("_WORLD")], tau=1.0)
    assert a.strings == b.strings and a.goto == b.goto and a.link == b.link
    assert np.array_equal(a.psi32, b.psi32) and np.array_equal(a.phi32, b.phi32)


def test_missing_character_piece_is_rejected():
    # 'b' appears only inside the piece "ab" (neither b nor B is a piece)
    vocab = [(0,), (0, 1)] + [(c,) for c in range(2, 53) if c != 28]
    with pytest.raises(ValueError):
        build_variative_graph(vocab, LOWER, [(0, 1)], tau=1.0)
