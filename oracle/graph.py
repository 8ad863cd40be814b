"""Oracle boosting graph for one phrase list — test infrastructure only.

Definitions (per model). Phrases p_i are token-id strings; cls maps every token
to its case class (Sec. II-A, case-insensitive matching: all case variants of a
token are one symbol). q_i = cls(p_i).

* F    = { q_i } (duplicates merged), Pref = every prefix of every q_i (the
         empty prefix is the root).
* States are the elements of Pref, numbered breadth first with children in
  ascending class order (root = 0).
* goto(x, c) = x.c when x.c is in Pref.
* link(x)    = the longest proper suffix of x that is in Pref (failure /
               suffix link, Sec. II-A and II-B "suffix-link targets").
* delta(s,c) = the state reached by the textbook Aho-Corasick move: follow
               links from s until a state with a c-child is found, else root.

Scores (Sec. II-A: potentials on states, an arc scores phi(dst) - phi(src)).
The paper leaves the numeric potentials of the tree open; the reading used
here ("commit", default) is:

* l(x)   = length of the longest prefix of x (x included) that is in F, else 0
* phi(x) = alpha * w * (|x| - l(x))                 pending partial-match score
* E(x)   = alpha * (w * (|x| - l(x[:-1])) + Bend)   if x in F
           alpha * Bend                              elif a proper suffix of x is in F
           0                                         otherwise
* psi(x) = phi(x) + E(x)

so a matched token earns w while the match is pending, completing a phrase
commits the pending score plus the end bonus, and breaking a match cancels
the pending part (step score phi(dst) - phi(src) + E(dst)).

The "pure_potential" reading: phi(x) = alpha*w*|x|, E(x) = alpha*Bend if some
suffix of x (x included) is in F.

All of phi, E, psi are computed in float64 from the strings themselves and
rounded once to float32.
"""

from __future__ import annotations

from collections import deque
from dataclasses import dataclass, field
from typing import Dict, List, Sequence, Tuple

import numpy as np

COMMIT = 0
PURE_POTENTIAL = 1


@dataclass
class Graph:
    strings: List[Tuple[int, ...]]          # state id -> class string
    goto: List[Dict[int, int]]              # state id -> {class: child id}
    link: List[int]                         # failure link (root -> 0)
    phi64: np.ndarray
    e64: np.ndarray
    psi64: np.ndarray
    phrases: frozenset                      # F
    class_map: np.ndarray                   # token -> class (blank -> -1)
    V: int                                  # blank id
    phi32: np.ndarray = None                # phi64, psi64 rounded once
    psi32: np.ndarray = None
    _rows: Dict[int, np.ndarray] = field(default_factory=dict)

    def __post_init__(self):
        self.phi32 = self.phi64.astype(np.float32)
        self.psi32 = self.psi64.astype(np.float32)

    @property
    def n_states(self) -> int:
        return len(self.strings)

    def delta(self, s: int, c: int) -> int:
        """Textbook Aho-Corasick move on class c from state s."""
        while True:
            if c in self.goto[s]:
                return self.goto[s][c]
            if s == 0:
                return 0
            s = self.link[s]

    def class_row(self, s: int) -> np.ndarray:
        """delta(s, c) for every class id c in [0, V) (memoised).

        The classic next-move table of Aho and Corasick: the row of a state is
        the row of its failure target, with the state's own children written
        over it; the root's row sends every class without a child to the root.
        """
        r = self._rows.get(s)
        if r is not None:
            return r
        if s == 0:
            r = np.zeros(self.V, dtype=np.int32)
        else:
            r = self.class_row(self.link[s]).copy()
        for c, y in self.goto[s].items():
            r[c] = y
        self._rows[s] = r
        return r

    def token_row(self, s: int) -> np.ndarray:
        """delta(s, cls v) for every non-blank token v (length V).

        A non-blank token without a class (class -1) matches nothing: its
        move goes to the root.
        """
        cm = self.class_map[: self.V]
        return np.where(cm >= 0, self.class_row(s)[np.maximum(cm, 0)], 0)


def _classes_of(tokens: Sequence[int], class_map: np.ndarray, V: int) -> Tuple[int, ...]:
    out = []
    for t in tokens:
        t = int(t)
        if t < 0 or t >= V:
            raise ValueError(f"token {t} outside [0, {V})")
        c = int(class_map[t])
        if c < 0:
            raise ValueError(f"token {t} has no class (blank cannot be in a phrase)")
        out.append(c)
    if not out:
        raise ValueError("empty phrase")
    return tuple(out)


def build_graph(phrase_tokens: Sequence[Sequence[int]], class_map: np.ndarray, *,
                token_w: float = 1.0, end_bonus: float = 2.0, alpha: float = 1.0,
                semantics: int = COMMIT) -> Graph:
    class_map = np.asarray(class_map)
    V = len(class_map) - 1
    F = frozenset(_classes_of(p, class_map, V) for p in phrase_tokens)

    # dictionary trie keyed by class strings
    trie: Dict[Tuple[int, ...], Dict[int, Tuple[int, ...]]] = {(): {}}
    for q in F:
        for i in range(1, len(q) + 1):
            pre = q[:i]
            if pre not in trie:
                trie[pre] = {}
                trie[q[:i - 1]][q[i - 1]] = pre

    # breadth-first numbering, children by ascending class
    strings: List[Tuple[int, ...]] = [()]
    ids = {(): 0}
    dq = deque([()])
    while dq:
        x = dq.popleft()
        for c in sorted(trie[x]):
            y = trie[x][c]
            ids[y] = len(strings)
            strings.append(y)
            dq.append(y)
    goto = [{c: ids[y] for c, y in trie[x].items()} for x in strings]

    # failure links, textbook breadth-first construction (Aho & Corasick 1975)
    link = [0] * len(strings)
    for sid, x in enumerate(strings):        # breadth-first order
        for c, y in sorted(goto[sid].items()):
            if sid == 0:
                link[y] = 0
                continue
            f = link[sid]
            while f != 0 and c not in goto[f]:
                f = link[f]
            link[y] = goto[f][c] if c in goto[f] and goto[f][c] != y else 0

    # potentials from the class strings themselves
    w, Bend, a = float(token_w), float(end_bonus), float(alpha)

    def ell(x):
        best = 0
        for i in range(1, len(x) + 1):
            if x[:i] in F:
                best = i
        return best

    n = len(strings)
    phi = np.zeros(n, dtype=np.float64)
    E = np.zeros(n, dtype=np.float64)
    for sid, x in enumerate(strings):
        if not x:
            continue
        if semantics == COMMIT:
            phi[sid] = a * w * (len(x) - ell(x))
            if x in F:
                E[sid] = a * (w * (len(x) - ell(x[:-1])) + Bend)
            elif any(x[i:] in F for i in range(1, len(x))):
                E[sid] = a * Bend
        elif semantics == PURE_POTENTIAL:
            phi[sid] = a * w * len(x)
            if any(x[i:] in F for i in range(0, len(x))):
                E[sid] = a * Bend
        else:
            raise ValueError("unknown semantics")
    return Graph(strings=strings, goto=goto, link=link, phi64=phi, e64=E,
                 psi64=phi + E, phrases=F, class_map=class_map, V=V)
