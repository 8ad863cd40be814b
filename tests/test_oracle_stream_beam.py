"""Pins of the oracle's streaming beam with recombination (Sec. II-C).

* without recombination it is the plain beam step;
* with every hypothesis kept, the merged score of a label sequence is the
  log of the summed probability of all its alignments (the forward sum over
  blank placements), found by enumerating every token sequence of a tiny
  vocabulary and grouping by label sequence;
* the flattened tree reproduces every slot's label sequence, and a tree of
  limited capacity marks the records it could not store;
* results do not depend on how the steps are split into calls.
"""

import itertools
import math

import numpy as np
import pytest
import scipy.special

import oracle
from oracle.graph import build_graph


def _cm(n):
    cm = np.arange(n + 1, dtype=np.int32)
    cm[n] = -1
    return cm


def _rows(seed, T, B, K, Vp1, scale=1.2):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((T, B, K, Vp1)) * scale).astype(np.float32)


def test_without_recombination_equals_the_plain_beam():
    cm = _cm(20)
    g = build_graph([[1, 2, 3], [2, 2], [5]], cm)
    rows = _rows(0, 30, 2, 4, 21)
    mids = [0, -1]
    st, S = oracle.init_carry(mids, 4)
    ref = oracle.beam_decode([g], mids, rows, st, S)
    carry = oracle.init_stream_carry(mids, 4)
    out = oracle.beam_decode_stream([g], mids, rows, carry, recombine=False)
    for a, b in zip(ref[:5], out[:5]):
        assert np.array_equal(a, b)
    assert np.array_equal(carry["states"], ref[5]) and np.array_equal(carry["scores"], ref[6])


@pytest.mark.parametrize("phrases", [[], [[0, 1]], [[1], [0, 0, 1]]])
@pytest.mark.parametrize("seed", range(3))
def test_merged_scores_are_forward_sums_over_alignments(phrases, seed):
    V, T = 2, 4
    cm = _cm(V)
    g = build_graph(phrases, cm)
    n_seq = sum((V) ** L for L in range(T + 1))       # label sequences of length <= T
    K = n_seq
    rows1 = _rows(seed, T, 1, 1, V + 1)[:, :, 0, :]
    rows = np.ascontiguousarray(np.repeat(rows1[:, :, None, :], K, axis=2))
    carry = oracle.init_stream_carry([0], K)
    out = oracle.beam_decode_stream([g], [0], rows, carry)
    # brute force: every token sequence, total log-prob + boost, grouped by labels
    lse = [scipy.special.logsumexp(rows1[t, 0].astype(np.float64)) for t in range(T)]
    groups = {}
    for seq in itertools.product(range(V + 1), repeat=T):
        s, tot, labels = 0, 0.0, []
        for t, v in enumerate(seq):
            tot += float(rows1[t, 0, v]) - lse[t]
            if v != V:
                ns = g.delta(s, int(cm[v]))
                tot += float(g.psi64[ns]) - float(g.phi64[s])
                s = ns
                labels.append(v)
        groups.setdefault(tuple(labels), []).append(tot)
    want = {k: scipy.special.logsumexp(v) for k, v in groups.items()}
    assert len(want) == n_seq
    got = {}
    for j in range(K):
        seq = oracle.tree_sequence(carry["trees"][0], int(carry["nodes"][0, j]))
        assert seq == carry["seqs"][0][j]
        got[seq] = float(carry["scores"][0, j])
    assert set(got) == set(want)
    for k in want:
        assert abs(got[k] - want[k]) < 2e-5 * max(1.0, abs(want[k])), (k, got[k], want[k])


def test_tree_records_and_capacity():
    cm = _cm(30)
    g = build_graph([[1, 2], [3, 4, 5]], cm)
    rows = _rows(4, 25, 2, 3, 31)
    carry = oracle.init_stream_carry([0, -1], 3)
    oracle.beam_decode_stream([g], [0, -1], rows, carry)
    for b in range(2):
        tree = carry["trees"][b]
        for node, (label, parent) in enumerate(tree):
            assert 0 <= label < 30 and -1 <= parent < node
        for j in range(3):
            assert oracle.tree_sequence(tree, int(carry["nodes"][b, j])) == carry["seqs"][b][j]
    small = oracle.init_stream_carry([0, -1], 3)
    oracle.beam_decode_stream([g], [0, -1], rows, small, tree_cap=10)
    assert all(len(t) == 10 for t in small["trees"])
    assert all(t == full[:10] for t, full in zip(small["trees"], carry["trees"]))
    assert np.any(small["nodes"] == -2)


def test_chunking_invariance():
    cm = _cm(16)
    g = build_graph([[1, 2, 3], [4, 4]], cm)
    rows = _rows(5, 33, 3, 4, 17, scale=0.8)
    mids = [0, 0, -1]
    full = oracle.init_stream_carry(mids, 4)
    ref = oracle.beam_decode_stream([g], mids, rows, full)
    part = oracle.init_stream_carry(mids, 4)
    outs = [oracle.beam_decode_stream([g], mids, rows[t0:t0 + 7], part) for t0 in range(0, 33, 7)]
    for i in range(5):
        assert np.array_equal(np.concatenate([o[i] for o in outs]), ref[i])
    assert part["trees"] == full["trees"] and np.array_equal(part["nodes"], full["nodes"])
