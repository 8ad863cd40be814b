"""Pins of the oracle's per-step fused score on biased streams.

The hand-derived worked examples (tests/golden/worked_example_*.txt) list, for
a few hypotheses, the boost of every step (the arc score phi(dst) - phi(src)
plus the end bonus of the state entered, Sec. II-A potentials). Here the
oracle's greedy and beam decoders are driven along each of those hypotheses
by giving the intended token a logit far above every other: the row's
log-softmax of that token is then exactly 0 in float32, so the emitted step
score must equal the golden boost exactly, and the emitted states the golden
states. Blank steps interleaved into a hypothesis must score 0 and keep the
state. A mistake in the score formula (for instance psi[dst] - psi[src], or
a dropped phi[src]) changes at least one of these numbers.
"""

import os

import numpy as np
import pytest

import oracle
from oracle.graph import COMMIT, PURE_POTENTIAL, build_graph
from tests import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
V = 8          # tokens 0..7 (token i is class i: letters a..e are 0..4), blank = 8
MARGIN = 60.0  # logit of the intended token; every other logit is 0


def _cm():
    cm = np.arange(V + 1, dtype=np.int32)
    cm[V] = -1
    return cm


def _forced_rows(seq):
    rows = np.zeros((len(seq), 1, V + 1), dtype=np.float32)
    for t, v in enumerate(seq):
        rows[t, 0, v] = MARGIN
    return rows


def _with_blanks(toks, boosts, sts):
    """Insert a blank after every token: (sequence, boosts, states)."""
    seq, bo, st = [], [], []
    for v, b, s in zip(toks, boosts, sts):
        seq += [v, V]
        bo += [b, 0.0]
        st += [s, s]
    return seq, bo, st


CASES = [("worked_example_commit.txt", COMMIT), ("worked_example_pure.txt", PURE_POTENTIAL)]


def test_margin_makes_log_softmax_zero():
    z = np.zeros(V + 1, dtype=np.float32)
    z[3] = MARGIN
    assert np.float32(z[3] - oracle.lse32(z)) == np.float32(0.0)


@pytest.mark.parametrize("fname,sem", CASES)
@pytest.mark.parametrize("blanks", [False, True])
def test_greedy_step_scores_follow_golden_boosts(fname, sem, blanks):
    phrases, w, B, _, hyps = brute.parse_golden(os.path.join(GOLDEN, fname))
    g = build_graph([list(p) for p in phrases], _cm(), token_w=w, end_bonus=B, semantics=sem)
    assert hyps
    for toks, boosts, sts in hyps:
        seq, bo, st = (_with_blanks(toks, boosts, sts) if blanks
                       else (list(toks), list(boosts), list(sts)))
        tok, ost, sc, fin = oracle.greedy_decode([g], [0], _forced_rows(seq),
                                                 np.zeros(1, np.int32))
        assert list(tok[:, 0]) == seq
        assert list(ost[:, 0]) == st
        assert [float(x) for x in sc[:, 0]] == bo
        assert fin[0] == st[-1]


@pytest.mark.parametrize("fname,sem", CASES)
@pytest.mark.parametrize("K", [1, 3])
def test_beam_step_scores_follow_golden_boosts(fname, sem, K):
    """The best beam hypothesis follows the forced path; its step scores are
    the golden boosts and its accumulated score is their running sum."""
    phrases, w, B, _, hyps = brute.parse_golden(os.path.join(GOLDEN, fname))
    g = build_graph([list(p) for p in phrases], _cm(), token_w=w, end_bonus=B, semantics=sem)
    for toks, boosts, sts in hyps:
        seq, bo, st = _with_blanks(toks, boosts, sts)
        rows = np.repeat(_forced_rows(seq)[:, :, None, :], K, axis=2)
        st0, S0 = oracle.init_carry([0], K)
        o_tok, o_par, o_st, o_step, o_cum, _, _ = oracle.beam_decode([g], [0], rows, st0, S0)
        # slot 0 is the best hypothesis; it extends the previous best (slot 0)
        assert list(o_tok[:, 0, 0]) == seq
        assert list(o_par[:, 0, 0]) == [0] * len(seq)
        assert list(o_st[:, 0, 0]) == st
        assert [float(x) for x in o_step[:, 0, 0]] == bo
        assert [float(x) for x in o_cum[:, 0, 0]] == list(np.cumsum(bo))


@pytest.mark.parametrize("alpha", [0.5, 2.0, 3.0])
def test_model_weight_scales_every_step_score(alpha):
    """The per-model boosting weight (Sec. II-B) multiplies every step boost."""
    phrases, w, B, _, hyps = brute.parse_golden(os.path.join(GOLDEN, "worked_example_commit.txt"))
    g = build_graph([list(p) for p in phrases], _cm(), token_w=w, end_bonus=B, alpha=alpha)
    for toks, boosts, sts in hyps:
        _, ost, sc, _ = oracle.greedy_decode([g], [0], _forced_rows(toks), np.zeros(1, np.int32))
        assert list(ost[:, 0]) == list(sts)
        assert [float(x) for x in sc[:, 0]] == [alpha * b for b in boosts]


def test_case_variant_scores_equal():
    """A case variant of a phrase token (same class, Sec. II-A) earns the same
    step score and reaches the same state as the canonical token."""
    phrases, w, B, _, hyps = brute.parse_golden(os.path.join(GOLDEN, "worked_example_commit.txt"))
    cm = _cm()
    cm[5], cm[6] = 0, 1          # tokens 5, 6 are case variants of a, b
    g = build_graph([list(p) for p in phrases], cm, token_w=w, end_bonus=B)
    swap = {0: 5, 1: 6}
    for toks, boosts, sts in hyps:
        seq = [swap.get(v, v) for v in toks]
        tok, ost, sc, _ = oracle.greedy_decode([g], [0], _forced_rows(seq), np.zeros(1, np.int32))
        assert list(tok[:, 0]) == seq
        assert list(ost[:, 0]) == list(sts)
        assert [float(x) for x in sc[:, 0]] == list(boosts)
