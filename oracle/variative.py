"""Oracle case-insensitive variative BPE graph (Sec. II-A, Fig. 1c and 1e,
Eq. (1)) — test infrastructure only.

Inputs: a piece vocabulary (token id -> string of character codes, cased), a
lowercasing map over character codes, and phrases as character strings.

Definitions (per model).

* canon(v)   = the lowercased character string of token v.
* cls(v)     = the smallest token id u with canon(u) = canon(v): one class per
               canonical string, so every cased spelling of a piece is one arc
               symbol (Sec. II-A).
* F          = the lowercased phrases (duplicates merged); Nodes = every prefix
               of every phrase, as character strings (the root is ()).
* arcs       : from node X there is an arc with class c exactly when
               X + canon(c) is a node (single-character pieces give the
               character chain, longer pieces the merged arcs; several arcs
               reach the same node, so the graph is a DAG).
* backbone   : the greedy tokenization of a lowercased phrase, read here as
               longest match from the left over the canonical strings.
* Eq. (1)    : the k-th backbone token, with score w and m_k characters,
               spreads w over its characters, the i-th getting
               w * exp((i+1)^tau) / sum_j exp((j+1)^tau).
* P(x)       = the cumulative score of prefix x along a phrase's backbone;
               a node shared by several phrases takes the largest.
* potentials ("commit" reading, as for the class graph, with |x| - l(x)
  replaced by the backbone score since the last completed phrase):
               l(x)   = length of the longest prefix of x (x included) in F
               phi(x) = alpha * (P(x) - P(x[:l(x)]))
               E(x)   = alpha * (P(x) - P(x[:l(x[:-1])]) + B)   if x in F
                        alpha * B              elif a proper suffix of x is in F
                        0                      otherwise
               psi    = phi + E
  "pure potential": phi = alpha * P(x), E = alpha * B if a suffix of x
  (x included) is in F.

Encoding as states (the step works on a tree-shaped record per arc):
every arc is a state whose target node it stands for; the root is state 0.
Nodes are expanded by increasing string length, nodes of one length in the
order of their first arc's id; expanding a node numbers its out-arcs
consecutively in ascending class order. Every arc into node T has T's out-arcs
as its children, T's potentials, and as suffix link the first arc into the
longest proper suffix of T that is a node (the root when none is).

The move on class c from a state standing for T goes to the arc (X, c) of
the longest suffix X of T (T included) that is a node with X + canon(c) a
node; to the root when there is none.
"""

from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple

import numpy as np

from .graph import COMMIT, PURE_POTENTIAL, Graph

Str = Tuple[int, ...]


def eq1_split(w: float, m: int, tau: float) -> List[float]:
    """Eq. (1): the shares of score w over the m characters of one token (float64)."""
    den = sum(math.exp(float(j + 1) ** tau) for j in range(m))
    return [w * math.exp(float(i + 1) ** tau) / den for i in range(m)]


def canon_strings(vocab: Sequence[Sequence[int]], lower: np.ndarray) -> List[Str]:
    return [tuple(int(lower[c]) for c in s) for s in vocab]


def class_map_of(vocab: Sequence[Sequence[int]], lower: np.ndarray) -> np.ndarray:
    """Token -> class (smallest token id with the same canonical string); blank -> -1."""
    can = canon_strings(vocab, lower)
    first: Dict[Str, int] = {}
    cm = np.full(len(vocab) + 1, -1, dtype=np.int32)
    for v, s in enumerate(can):
        if not s:
            raise ValueError(f"token {v} has an empty string")
        first.setdefault(s, v)
        cm[v] = first[s]
    return cm


def greedy_backbone(phrase: Str, pieces: set) -> List[int]:
    """Longest-match tokenization of a lowercased phrase: the lengths m_k."""
    out, i = [], 0
    longest = max(len(p) for p in pieces)
    while i < len(phrase):
        for m in range(min(longest, len(phrase) - i), 0, -1):
            if phrase[i:i + m] in pieces:
                out.append(m)
                i += m
                break
        else:
            raise ValueError(f"character {phrase[i]} is not a piece of the vocabulary")
    return out


def build_variative_graph(vocab: Sequence[Sequence[int]], lower: np.ndarray,
                          phrases: Sequence[Sequence[int]], *, token_w: float = 1.0,
                          end_bonus: float = 2.0, alpha: float = 1.0, tau: float = 1.0,
                          semantics: int = COMMIT) -> Graph:
    lower = np.asarray(lower)
    V = len(vocab)
    cm = class_map_of(vocab, lower)
    can = canon_strings(vocab, lower)
    class_str: Dict[int, Str] = {int(cm[v]): can[v] for v in range(V)}
    pieces = set(can)
    F = frozenset(tuple(int(lower[c]) for c in p) for p in phrases)
    if any(len(p) == 0 for p in F):
        raise ValueError("empty phrase")
    # the character chain needs every character as a piece of its own
    for p in F:
        for ch in p:
            if (ch,) not in pieces:
                raise ValueError(f"character {ch} is not a single-character piece")

    # nodes and their backbone potentials (largest over the phrases through them)
    w, Bend, a = float(token_w), float(end_bonus), float(alpha)
    P: Dict[Str, float] = {(): 0.0}
    for p in sorted(F):
        acc, pos = 0.0, 0
        for m in greedy_backbone(p, pieces):
            for d in eq1_split(w, m, float(tau)):
                acc += d
                pos += 1
                P[p[:pos]] = max(P.get(p[:pos], -math.inf), acc)
    nodes = set(P)

    # arcs: X --c--> X + canon(c) whenever that is a node
    out_arcs: Dict[Str, List[Tuple[int, Str]]] = {}
    for X in nodes:
        out_arcs[X] = sorted((c, X + s) for c, s in class_str.items() if X + s in nodes)

    # numbering: nodes by length, then by the id of their first arc
    ids_of: Dict[Str, int] = {(): 0}          # node -> first arc (state) into it
    target: List[Str] = [()]                   # state -> node
    block: Dict[Str, Tuple[int, int]] = {}     # node -> (first child, count)
    for L in range(0, max(len(x) for x in nodes) + 1):
        for X in sorted((x for x in nodes if len(x) == L), key=lambda x: ids_of[x]):
            first = len(target)
            for c, T in out_arcs[X]:
                if T not in ids_of:
                    ids_of[T] = len(target)
                target.append(T)
            block[X] = (first, len(out_arcs[X]))

    def suffix_node(T: Str) -> Str:
        for i in range(1, len(T) + 1):
            if T[i:] in nodes:
                return T[i:]
        return ()

    n = len(target)
    goto = [{c: block[T][0] + j for j, (c, _) in enumerate(out_arcs[T])} for T in target]
    link = [ids_of[suffix_node(T)] if T else 0 for T in target]

    def ell(x: Str) -> int:
        best = 0
        for i in range(1, len(x) + 1):
            if x[:i] in F:
                best = i
        return best

    phi = np.zeros(n, dtype=np.float64)
    E = np.zeros(n, dtype=np.float64)
    for sid, x in enumerate(target):
        if not x:
            continue
        if semantics == COMMIT:
            phi[sid] = a * (P[x] - P[x[:ell(x)]])
            if x in F:
                E[sid] = a * ((P[x] - P[x[:ell(x[:-1])]]) + Bend)
            elif any(x[i:] in F for i in range(1, len(x))):
                E[sid] = a * Bend
        elif semantics == PURE_POTENTIAL:
            phi[sid] = a * P[x]
            if any(x[i:] in F for i in range(0, len(x))):
                E[sid] = a * Bend
        else:
            raise ValueError("unknown semantics")
    return Graph(strings=target, goto=goto, link=link, phi64=phi, e64=E, psi64=phi + E,
                 phrases=F, class_map=cm, V=V)


def move_by_strings(g: Graph, vocab, lower, s: int, v: int) -> int:
    """The move on token v from state s, from the strings alone: the arc
    (X, cls v) of the longest suffix X of s's node with X + canon(v) a node."""
    can = tuple(int(lower[c]) for c in vocab[v])
    c = int(g.class_map[v])
    T = g.strings[s]
    nodes = set(g.strings)
    for i in range(0, len(T) + 1):
        X = T[i:]
        if X in nodes and X + can in nodes:
            # the arc (X, c): the child of any state standing for X on class c
            sx = g.strings.index(X)
            return g.goto[sx][c]
    return 0
