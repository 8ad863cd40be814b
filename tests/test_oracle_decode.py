"""Pins of the oracle greedy and beam steps against things other than itself.

* log-sum-exp: closed form for a constant row, and scipy's logsumexp;
* greedy: brute-force keys z[v] + psi(sigma(h.v)) with sigma found by suffix
  enumeration over the whole history, selection by sorting;
* beam: with K at least the number of live hypotheses, beam search equals
  exhaustive enumeration of every token sequence (totals recomputed from
  scratch); model -1 equals textbook beam search on log-softmax scores;
* invariants stated by the paper: model -1 decodes exactly as an unbiased
  stream, streams are isolated, results do not depend on chunking (Sec. II-B,
  II-C), case variants are interchangeable (Sec. II-A).
"""

import itertools
import math

import numpy as np
import pytest
import scipy.special

import oracle
from oracle.graph import build_graph
from tests import brute


def _cm(n):
    cm = np.arange(n + 1, dtype=np.int32)
    cm[n] = -1
    return cm


def test_lse_closed_form_constant_row():
    for c, n in [(0.0, 257), (3.5, 1025), (-7.25, 8193)]:
        z = np.full(n, c, dtype=np.float32)
        assert oracle.lse32(z) == np.float32(c + math.log(n))


def test_lse_matches_scipy():
    rng = np.random.default_rng(0)
    for n in (2, 257, 1025, 8193):
        for _ in range(20):
            z = (rng.standard_normal(n) * rng.uniform(0.1, 20)).astype(np.float32)
            ref = scipy.special.logsumexp(z.astype(np.float64))
            got = oracle.lse32(z)
            assert abs(float(got) - ref) <= 0.5 * float(np.spacing(np.float32(abs(ref)))) + 1e-12


def _brute_greedy(F, cm, g, rows):
    """Greedy decoding from scratch: sigma by suffix enumeration, psi/phi read
    off the (golden-pinned) per-state potentials by state string."""
    pref = brute.prefixes(F)
    by_string = {x: i for i, x in enumerate(g.strings)}
    V = rows.shape[1] - 1
    hist = []
    toks = []
    for z in rows:
        s_str = brute.sigma(hist, pref)
        s = by_string[s_str]
        keys = []
        for v in range(V + 1):
            if v == V:
                k = np.float32(z[V] + g.phi32[s])
            else:
                d = by_string[brute.sigma(hist + [int(cm[v])], pref)]
                k = np.float32(z[v] + g.psi32[d])
            keys.append((k, v))
        best = sorted(keys, key=lambda kv: (-kv[0], kv[1]))[0][1]
        toks.append(best)
        if best != V:
            hist.append(int(cm[best]))
    return toks


@pytest.mark.parametrize("seed", range(6))
def test_greedy_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    from workloads import Config, class_map
    cfg = Config(0, "t", B=1, K=1, V=12, T=1, chunk=1, dtype="f32", n_phrases=0, len_lo=1,
                 len_hi=1, token_dist="uniform", zipf_s=0, logit_std=1, blank_offset=0, n_case=3)
    cm = class_map(cfg)
    phrases = [list(rng.integers(0, 12, size=rng.integers(1, 4))) for _ in range(5)]
    F = [tuple(int(cm[t]) for t in p) for p in phrases]
    g = build_graph(phrases, cm)
    T = 40
    # logits favouring phrase tokens so that matches happen
    rows = rng.standard_normal((T, 13)).astype(np.float32)
    rows[:, :9] += np.float32(0.8)
    tok, st, sc, fin = oracle.greedy_decode([g], [0], rows[:, None, :], np.zeros(1, np.int32))
    assert list(tok[:, 0]) == _brute_greedy(F, cm, g, rows)


def test_greedy_ties_go_to_lowest_index():
    cm = _cm(6)
    g = build_graph([[3]], cm)   # token 3 gets psi = w + B = 3
    z = np.zeros((1, 1, 7), dtype=np.float32)
    z[0, 0, 3] = 1.0             # key 4
    z[0, 0, 5] = 4.0             # key 4 as well; lower index 3 wins
    z[0, 0, 6] = 4.0             # blank key 4
    tok, st, sc, _ = oracle.greedy_decode([g], [0], z, np.zeros(1, np.int32))
    assert tok[0, 0] == 3 and st[0, 0] == 1


def test_model_minus_one_is_unbiased():
    rng = np.random.default_rng(3)
    rows = rng.standard_normal((30, 1, 65)).astype(np.float32)
    g = build_graph([[1, 2], [3]], _cm(64))
    tok, st, sc, fin = oracle.greedy_decode([g], [-1], rows, np.full(1, -1, np.int32))
    assert np.array_equal(tok[:, 0], np.argmax(rows[:, 0], axis=1))
    assert np.all(st == -1) and fin[0] == -1
    lse = scipy.special.logsumexp(rows[:, 0].astype(np.float64), axis=1)
    zsel = rows[np.arange(30), 0, tok[:, 0]]
    assert np.allclose(sc[:, 0], zsel - lse, atol=2e-6)


def _exhaustive(F, cm, g, rows):
    """Every token sequence with its total score, recomputed from scratch (float64)."""
    pref = brute.prefixes(F)
    by_string = {x: i for i, x in enumerate(g.strings)}
    T, Vp1 = rows.shape
    V = Vp1 - 1
    lse = [scipy.special.logsumexp(r.astype(np.float64)) for r in rows]
    out = []
    for seq in itertools.product(range(Vp1), repeat=T):
        hist, tot = [], 0.0
        for t, v in enumerate(seq):
            s = by_string[brute.sigma(hist, pref)]
            if v == V:
                b = 0.0
            else:
                hist.append(int(cm[v]))
                d = by_string[brute.sigma(hist, pref)]
                b = float(g.psi64[d]) - float(g.phi64[s])
            tot += float(rows[t, v]) - lse[t] + b
        out.append((tot, seq))
    out.sort(key=lambda x: -x[0])
    return out


def _backtrack(tok, par, j):
    T = tok.shape[0]
    seq = []
    for t in range(T - 1, -1, -1):
        seq.append(int(tok[t, j]))
        j = int(par[t, j])
    return tuple(reversed(seq))


@pytest.mark.parametrize("seed", range(5))
def test_beam_equals_exhaustive_search(seed):
    rng = np.random.default_rng(seed)
    V, T = 3, 3
    cm = _cm(V)
    phrases = [[0, 1], [1], [2, 2, 0]][: 1 + seed % 3]
    F = [tuple(p) for p in phrases]
    g = build_graph(phrases, cm)
    rows = (rng.standard_normal((T, V + 1)) * 1.5).astype(np.float32)
    K = (V + 1) ** (T - 1)       # keeps every live hypothesis until the last step
    rk = np.repeat(rows[:, None, None, :], K, axis=2)
    st, S = oracle.init_carry([0], K)
    tok, par, ost, step, cum, _, _ = oracle.beam_decode([g], [0], rk, st, S)
    ex = _exhaustive(F, cm, g, rows)
    for j in range(K):
        assert abs(float(cum[-1, 0, j]) - ex[j][0]) < 1e-4
        if j + 1 < K and ex[j][0] - ex[j + 1][0] > 1e-4 and (j == 0 or ex[j - 1][0] - ex[j][0] > 1e-4):
            assert _backtrack(tok[:, 0], par[:, 0], j) == ex[j][1]


def test_beam_model_minus_one_is_textbook_beam():
    rng = np.random.default_rng(7)
    T, K, Vp1 = 12, 4, 33
    rows = rng.standard_normal((T, 1, K, Vp1)).astype(np.float32)
    st, S = oracle.init_carry([-1], K)
    tok, par, ost, step, cum, _, _ = oracle.beam_decode([], [-1], rows, st, S)
    # textbook: score every extension by its log-softmax, keep the K best
    hyps = [(0.0, [])] + [(-math.inf, [])] * (K - 1)
    for t in range(T):
        cand = []
        for k, (sc, seq) in enumerate(hyps):
            lp = rows[t, 0, k].astype(np.float64) - scipy.special.logsumexp(
                rows[t, 0, k].astype(np.float64))
            for v in range(Vp1):
                cand.append((sc + lp[v], k * Vp1 + v, seq + [v]))
        cand.sort(key=lambda x: (-x[0], x[1]))
        hyps = [(c[0], c[2]) for c in cand[:K]]
        assert np.allclose(cum[t, 0], [h[0] for h in hyps], atol=1e-4)
    assert np.all(ost == -1)
    for j in range(K):
        assert list(_backtrack(tok[:, 0], par[:, 0], j)) == hyps[j][1]


def _setup(seed, B=4, V=40, n_case=5, T=30):
    from workloads import Config, class_map
    cfg = Config(0, "t", B=B, K=1, V=V, T=T, chunk=T, dtype="f32", n_phrases=0, len_lo=1,
                 len_hi=1, token_dist="uniform", zipf_s=0, logit_std=1, blank_offset=0,
                 n_case=n_case)
    cm = class_map(cfg)
    rng = np.random.default_rng(seed)
    graphs = [build_graph([list(rng.integers(0, 15, size=rng.integers(1, 4))) for _ in range(6)], cm)
              for _ in range(B)]
    rows = rng.standard_normal((T, B, V + 1)).astype(np.float32)
    rows[:, :, :15] += np.float32(0.7)
    return cfg, cm, graphs, rows


def test_stream_isolation_and_permutation():
    cfg, cm, graphs, rows = _setup(1)
    B = cfg.B
    mids = list(range(B))
    st0 = np.zeros(B, np.int32)
    ref = oracle.greedy_decode(graphs, mids, rows, st0)
    perm = np.array([2, 0, 3, 1])
    out = oracle.greedy_decode(graphs, [mids[p] for p in perm], rows[:, perm], st0[perm])
    for a, b in zip(ref[:3], out[:3]):
        assert np.array_equal(a[:, perm], b)
    # changing stream 1's list leaves the others bit-identical
    g2 = list(graphs)
    g2[1] = build_graph([[0, 1, 2, 3]], cm)
    out2 = oracle.greedy_decode(g2, mids, rows, st0)
    for a, b in zip(ref[:3], out2[:3]):
        assert np.array_equal(a[:, [0, 2, 3]], b[:, [0, 2, 3]])


def test_chunking_invariance():
    cfg, cm, graphs, rows = _setup(2)
    B, T = cfg.B, cfg.T
    mids = list(range(B))
    full = oracle.greedy_decode(graphs, mids, rows, np.zeros(B, np.int32))
    for ch in (1, 7, 16):
        st = np.zeros(B, np.int32)
        parts = []
        for t0 in range(0, T, ch):
            r = oracle.greedy_decode(graphs, mids, rows[t0:t0 + ch], st)
            parts.append(r)
            st = r[3]
        for i in range(3):
            assert np.array_equal(np.concatenate([p[i] for p in parts]), full[i])
    # beam
    K = 3
    rk = np.repeat(rows[:, :, None, :], K, axis=2)
    st, S = oracle.init_carry(mids, K)
    fullb = oracle.beam_decode(graphs, mids, rk, st, S)
    st, S = oracle.init_carry(mids, K)
    parts = []
    for t0 in range(0, T, 7):
        r = oracle.beam_decode(graphs, mids, rk[t0:t0 + 7], st, S)
        parts.append(r)
        st, S = r[5], r[6]
    for i in range(5):
        assert np.array_equal(np.concatenate([p[i] for p in parts]), fullb[i])


def test_case_swap_of_logit_columns():
    """Swapping the logits of two case variants swaps the emitted variant only."""
    cfg, cm, graphs, rows = _setup(4)
    n = cfg.n_case
    B = cfg.B
    mids = list(range(B))
    ref = oracle.greedy_decode(graphs, mids, rows, np.zeros(B, np.int32))
    sw = rows.copy()
    for c in range(n):
        sw[:, :, [c, c + n]] = rows[:, :, [c + n, c]]
    out = oracle.greedy_decode(graphs, mids, sw, np.zeros(B, np.int32))
    mapping = np.arange(cfg.V + 1)
    for c in range(n):
        mapping[c], mapping[c + n] = c + n, c
    # states and scores are unchanged unless a tie between variants decides differently
    assert np.array_equal(out[1], ref[1])
    assert np.array_equal(out[0], mapping[ref[0]])
    assert np.array_equal(out[2], ref[2])
