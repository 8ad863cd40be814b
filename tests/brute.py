"""Brute-force references for tiny inputs (test helpers; no oracle code).

Everything here works on whole hypothesis strings by enumeration, never by the
incremental automaton: sigma(h) is found by trying every suffix of h.
"""

from __future__ import annotations

import itertools
from typing import Dict, Iterable, List, Sequence, Set, Tuple


def prefixes(F: Iterable[Tuple[int, ...]]) -> Set[Tuple[int, ...]]:
    out = {()}
    for f in F:
        for i in range(1, len(f) + 1):
            out.add(tuple(f[:i]))
    return out


def sigma(h: Sequence[int], pref: Set[Tuple[int, ...]]) -> Tuple[int, ...]:
    """Longest suffix of h that is a phrase prefix (the graph state after h)."""
    h = tuple(h)
    for i in range(len(h) + 1):
        if h[i:] in pref:
            return h[i:]
    return ()


def all_strings(n_sym: int, max_len: int):
    for L in range(max_len + 1):
        yield from itertools.product(range(n_sym), repeat=L)


def parse_golden(path: str):
    """Parse a worked-example fixture (tests/golden/worked_example_*.txt)."""
    letters = "abcde"
    phrases: List[Tuple[int, ...]] = []
    states = []
    hyps = []
    w = B = None
    with open(path) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, _, rest = line.partition(":")
            rest = rest.strip()
            if key == "phrases":
                phrases = [tuple(letters.index(ch) for ch in p) for p in rest.split()]
            elif key == "w":
                w = float(rest)
            elif key == "B":
                B = float(rest)
            elif key == "state":
                sid, s, link, phi, E, psi = rest.split()
                string = () if s == "-" else tuple(letters.index(ch) for ch in s)
                states.append((int(sid), string, int(link), float(phi), float(E), float(psi)))
            elif key == "hyp":
                toks, _, tail = rest.partition("->")
                boosts, _, sts = tail.partition(";")
                hyps.append((tuple(letters.index(ch) for ch in toks.strip()),
                             [float(x) for x in boosts.split()], [int(x) for x in sts.split()]))
    return phrases, w, B, states, hyps
