"""Oracle boosted greedy and beam steps — test infrastructure only.

One step of a stream (Sec. II-B, fused scoring operation): for every token v,
the boosting score of v from the stream's current graph state s is added to
the joint logit z_v; the stream then selects (argmax for greedy, top-K over
all K*(V+1) extensions for beam) and advances its graph state. Model id -1
means no biasing: the boost is zero and the state stays -1 (Sec. II-B).

Per row, in float32 with this exact operation order:

* key[v]     = z[v] + psi[delta(s, cls v)]      for v < V
* key[V]     = z[V] + phi[s]                     (blank: no advance)
  (subtracting phi[s] from every key gives the step boost
   b = phi(dst) - phi(s) + E(dst); keeping it out of the key leaves the
   selection unchanged and keeps the key one rounding away from z)
* lse        = max z + log(sum exp(z - max z)), sum and log in float64,
               rounded once to float32 (log-softmax normalizer)
* greedy     : v* = first index of the maximum key (ties -> lowest v)
* beam       : c_k  = (S_k - lse_k) - phi[s_k];  cand = c_k + key_k[v];
               keep the K largest cand over the flat index k*(V+1)+v,
               sorted descending, ties -> lowest flat index
* step score : (z[v] - lse) + b with b = psi[dst] - phi[s] (0 for blank)

Model -1 uses phi = psi = 0 and keeps state -1.
"""

from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .graph import Graph


def widen(rows: np.ndarray) -> np.ndarray:
    """float32 rows as they are; uint16 bfloat16 bits widened exactly."""
    if rows.dtype == np.float32:
        return rows
    if rows.dtype == np.uint16:
        return (rows.astype(np.uint32) << np.uint32(16)).view(np.float32)
    raise TypeError(rows.dtype)


def lse32(z: np.ndarray) -> np.float32:
    """log(sum(exp(z))) of one float32 row: float64 exact sum, one rounding."""
    m = float(np.max(z))
    s = math.fsum(np.exp(z.astype(np.float64) - m).tolist())
    return np.float32(m + math.log(s))


def _keys(g: Optional[Graph], s: int, z: np.ndarray):
    """(key[V+1], dst[V] or None, phi_s) for state s; float32 keys."""
    V = z.shape[0] - 1
    if g is None:
        return z.copy(), None, np.float32(0.0)
    dst = g.token_row(s)
    psi = g.psi32
    phi_s = g.phi32[s]
    key = np.empty(V + 1, dtype=np.float32)
    key[:V] = z[:V] + psi[dst]
    key[V] = z[V] + phi_s
    return key, dst, phi_s


def _boost(g: Optional[Graph], s: int, v: int, dst_state: int, V: int) -> np.float32:
    if g is None or v == V:
        return np.float32(0.0)
    return np.float32(g.psi32[dst_state] - g.phi32[s])


def init_carry(model_ids: Sequence[int], K: int = 1):
    """Initial states (0, or -1 for model -1) and beam scores [0, -inf, ...]."""
    B = len(model_ids)
    st = np.zeros((B, K), dtype=np.int32)
    for b, m in enumerate(model_ids):
        if m < 0:
            st[b, :] = -1
    S = np.full((B, K), -np.inf, dtype=np.float32)
    S[:, 0] = 0.0
    return st, S


def greedy_decode(graphs: Sequence[Graph], model_ids: Sequence[int], rows: np.ndarray,
                  states: np.ndarray, streams: Optional[Sequence[int]] = None):
    """Greedy boosted decoding of rows [T, B, V+1] (or [T, B, 1, V+1]).

    ``states`` [B] is the carried state (updated copy returned). ``streams``
    restricts the work to a subset of the B streams (others are left untouched
    and their outputs are zero). Returns (tok, state, score, states_out) with
    shapes [T, B].
    """
    rows = np.asarray(rows)
    if rows.ndim == 4:
        rows = rows[:, :, 0, :]
    T, B, Vp1 = rows.shape
    V = Vp1 - 1
    states = np.asarray(states, dtype=np.int32).reshape(B).copy()
    tok = np.zeros((T, B), dtype=np.int32)
    st = np.zeros((T, B), dtype=np.int32)
    sc = np.zeros((T, B), dtype=np.float32)
    for b in (range(B) if streams is None else streams):
        m = int(model_ids[b])
        g = graphs[m] if m >= 0 else None
        s = int(states[b])
        for t in range(T):
            z = widen(rows[t, b])
            lse = lse32(z)
            key, dst, _ = _keys(g, s, z)
            v = int(np.argmax(key))          # first maximum
            if g is None:
                ns = -1
            elif v == V:
                ns = s
            else:
                ns = int(dst[v])
            b_ = _boost(g, s, v, ns, V)
            tok[t, b] = v
            st[t, b] = ns
            sc[t, b] = np.float32(np.float32(z[v] - lse) + b_)
            s = ns
        states[b] = s
    return tok, st, sc, states


def beam_decode(graphs: Sequence[Graph], model_ids: Sequence[int], rows: np.ndarray,
                states: np.ndarray, scores: np.ndarray,
                streams: Optional[Sequence[int]] = None):
    """Beam boosted decoding of rows [T, B, K, V+1] with carry states/scores [B, K].

    Returns (tok, parent, state, step, cum, states_out, scores_out); the
    per-step arrays have shape [T, B, K].
    """
    rows = np.asarray(rows)
    T, B, K, Vp1 = rows.shape
    V = Vp1 - 1
    states = np.asarray(states, dtype=np.int32).reshape(B, K).copy()
    scores = np.asarray(scores, dtype=np.float32).reshape(B, K).copy()
    o_tok = np.zeros((T, B, K), dtype=np.int32)
    o_par = np.zeros((T, B, K), dtype=np.int32)
    o_st = np.zeros((T, B, K), dtype=np.int32)
    o_step = np.zeros((T, B, K), dtype=np.float32)
    o_cum = np.zeros((T, B, K), dtype=np.float32)
    flat_idx = np.arange(K * Vp1)
    for b in (range(B) if streams is None else streams):
        m = int(model_ids[b])
        g = graphs[m] if m >= 0 else None
        for t in range(T):
            cands = np.empty(K * Vp1, dtype=np.float32)
            info = []
            for k in range(K):
                s = int(states[b, k])
                z = widen(rows[t, b, k])
                lse = lse32(z)
                key, dst, phi_s = _keys(g, s, z)
                c_k = np.float32(np.float32(scores[b, k] - lse) - phi_s)
                cands[k * Vp1:(k + 1) * Vp1] = c_k + key
                info.append((s, z, lse, dst))
            order = np.lexsort((flat_idx, -cands))[:K]
            new_st = np.empty(K, dtype=np.int32)
            new_sc = np.empty(K, dtype=np.float32)
            for j, f in enumerate(order):
                k, v = divmod(int(f), Vp1)
                s, z, lse, dst = info[k]
                if g is None:
                    ns = -1
                elif v == V:
                    ns = s
                else:
                    ns = int(dst[v])
                b_ = _boost(g, s, v, ns, V)
                o_tok[t, b, j] = v
                o_par[t, b, j] = k
                o_st[t, b, j] = ns
                o_step[t, b, j] = np.float32(np.float32(z[v] - lse) + b_)
                o_cum[t, b, j] = cands[f]
                new_st[j] = ns
                new_sc[j] = cands[f]
            states[b] = new_st
            scores[b] = new_sc
    return o_tok, o_par, o_st, o_step, o_cum, states, scores


# ---------------------------------------------------------------------------
# Streaming beam search with hypothesis recombination and a flattened
# hypothesis tree (Sec. II-C: finalized hypotheses are kept in a flattened tree
# with their accumulated scores, and are continued, merged and pruned across
# chunks).
#
# A hypothesis is its label sequence (the emitted non-blank tokens). Two
# candidates of a step are the same hypothesis when their label sequences are
# equal; they are merged into one candidate whose score is the log of the sum
# of their probabilities (float64 log-add-exp of the two float32 scores,
# rounded once to float32). The merged candidate keeps the position (slot and
# token) of the better of the two in (score descending, flat index ascending)
# order; the other is dropped. Only finite candidates of live slots (finite
# accumulated score) are merged. Because the live slots of a step hold
# distinct label sequences, a duplicate pair is always
# "slot i extended by the blank" with "slot j extended by the last label of
# slot i" where slot j holds slot i's sequence without its last label.
#
# The tree holds one record (label, parent record) per non-blank extension
# that was kept, appended in slot order after every step; a slot's node is the
# record of its last label (-1 for the empty sequence). A record that does
# not fit the stream's capacity is not stored and its node is -2.


def init_stream_carry(model_ids: Sequence[int], K: int):
    """Carry of the streaming beam: states, scores, label sequences, nodes, trees."""
    st, S = init_carry(model_ids, K)
    B = len(model_ids)
    return {"states": st, "scores": S, "seqs": [[()] * K for _ in range(B)],
            "nodes": np.full((B, K), -1, np.int32), "trees": [[] for _ in range(B)]}


def _logaddexp32(a: np.float32, b: np.float32) -> np.float32:
    return np.float32(np.logaddexp(np.float64(a), np.float64(b)))


def beam_decode_stream(graphs, model_ids: Sequence[int], rows: np.ndarray, carry: dict,
                       recombine: bool = True, tree_cap: Optional[int] = None):
    """Streaming beam over rows [T, B, K, V+1] with the carry of init_stream_carry
    (updated in place and returned). Per-step outputs as beam_decode's."""
    rows = np.asarray(rows)
    T, B, K, Vp1 = rows.shape
    V = Vp1 - 1
    states, scores = carry["states"], carry["scores"]
    seqs, nodes, trees = carry["seqs"], carry["nodes"], carry["trees"]
    o_tok = np.zeros((T, B, K), dtype=np.int32)
    o_par = np.zeros((T, B, K), dtype=np.int32)
    o_st = np.zeros((T, B, K), dtype=np.int32)
    o_step = np.zeros((T, B, K), dtype=np.float32)
    o_cum = np.zeros((T, B, K), dtype=np.float32)
    flat_idx = np.arange(K * Vp1)
    for b in range(B):
        m = int(model_ids[b])
        g = graphs[m] if m >= 0 else None
        for t in range(T):
            cands = np.empty(K * Vp1, dtype=np.float32)
            info = []
            for k in range(K):
                s = int(states[b, k])
                z = widen(rows[t, b, k])
                lse = lse32(z)
                key, dst, phi_s = _keys(g, s, z)
                c_k = np.float32(np.float32(scores[b, k] - lse) - phi_s)
                cands[k * Vp1:(k + 1) * Vp1] = c_k + key
                info.append((s, z, lse, dst))
            if recombine:
                for i in range(K):
                    if not seqs[b][i] or not np.isfinite(scores[b, i]):
                        continue
                    for j in range(K):
                        if j != i and np.isfinite(scores[b, j]) and seqs[b][j] == seqs[b][i][:-1]:
                            v = seqs[b][i][-1]
                            fa, fb = i * Vp1 + V, j * Vp1 + v
                            a, c = cands[fa], cands[fb]
                            if np.isfinite(a) and np.isfinite(c):
                                merged = _logaddexp32(a, c)
                                keep_a = a > c or (a == c and fa < fb)
                                cands[fa if keep_a else fb] = merged
                                cands[fb if keep_a else fa] = -np.inf
                            break
            order = np.lexsort((flat_idx, -cands))[:K]
            new_st = np.empty(K, dtype=np.int32)
            new_sc = np.empty(K, dtype=np.float32)
            new_seq, new_node = [], np.empty(K, dtype=np.int32)
            for j, f in enumerate(order):
                k, v = divmod(int(f), Vp1)
                s, z, lse, dst = info[k]
                if g is None:
                    ns = -1
                elif v == V:
                    ns = s
                else:
                    ns = int(dst[v])
                b_ = _boost(g, s, v, ns, V)
                o_tok[t, b, j] = v
                o_par[t, b, j] = k
                o_st[t, b, j] = ns
                o_step[t, b, j] = np.float32(np.float32(z[v] - lse) + b_)
                o_cum[t, b, j] = cands[f]
                new_st[j] = ns
                new_sc[j] = cands[f]
                if v == V:
                    new_seq.append(seqs[b][k])
                    new_node[j] = nodes[b, k]
                else:
                    new_seq.append(seqs[b][k] + (v,))
                    if tree_cap is not None and len(trees[b]) >= tree_cap:
                        new_node[j] = -2
                    else:
                        new_node[j] = len(trees[b])
                        trees[b].append((v, int(nodes[b, k])))
            states[b] = new_st
            scores[b] = new_sc
            seqs[b] = new_seq
            nodes[b] = new_node
    return o_tok, o_par, o_st, o_step, o_cum, carry


def tree_sequence(tree, node: int) -> Tuple[int, ...]:
    """Label sequence of a tree node (following parent records to the root)."""
    out = []
    while node >= 0:
        label, node = tree[node]
        out.append(label)
    return tuple(reversed(out))
