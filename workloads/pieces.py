"""Synthetic piece vocabulary, character-coded phrase lists and logits for the
variative BPE graph (Sec. II-A, Fig. 1c/1e).

No tokenizer or text is available, so the vocabulary is drawn from a seeded
random lexicon:

* characters: 0..25 lowercase letters, 26 the word-start mark, 27..52 the
  uppercase letters (their lowercase is code - 27);
* tokens 0..52 are the single characters (every character is a piece, as in
  a SentencePiece vocabulary built from character pieces); the rest are the
  most frequent word-initial and word-internal substrings (2..6 characters)
  of the lexicon, some of them with a Title or UPPER spelling as well (a piece
  may exist in one casing and not in another);
* a phrase is one to three lexicon words, each with the word-start mark and a
  random casing;
* logits are N(0, std) with a blank offset; in every slot of 16 steps one
  phrase of the stream is planted, spelled by a random segmentation into
  pieces and a random casing of each piece.

This module only draws random numbers and lays out inputs; the graph
construction and its scores are not here.
"""

from __future__ import annotations

from collections import Counter
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .synth import Config, _f32_to_bf16_bits

N_CHARS = 53
WORD = 26
LOWER = np.array(list(range(27)) + list(range(26)), dtype=np.int32)


@dataclass(frozen=True)
class PieceConfig:
    index: int
    name: str
    B: int
    K: int
    V: int              # non-blank tokens (pieces); blank id = V
    T: int
    chunk: int
    dtype: str
    n_phrases: int
    words_lo: int = 1
    words_hi: int = 3
    n_lexicon: int = 3000
    title_frac: float = 0.3
    upper_frac: float = 0.1
    logit_std: float = 1.0
    blank_offset: float = 1.5
    plant_boost: float = 4.0
    tau: float = 1.0
    token_w: float = 1.0
    end_bonus: float = 2.0

    @property
    def Vp1(self) -> int:
        return self.V + 1


PIECE_CONFIGS = (
    PieceConfig(20, "variative_small", B=8, K=1, V=400, T=96, chunk=16, dtype="f32",
                n_phrases=40, n_lexicon=400),
    PieceConfig(21, "variative_streaming", B=128, K=1, V=1024, T=1024, chunk=16, dtype="f32",
                n_phrases=1000),
)


def piece_config(name: str, **kw) -> PieceConfig:
    from dataclasses import replace
    for c in PIECE_CONFIGS:
        if c.name == name:
            return replace(c, **kw) if kw else c
    raise KeyError(name)


def _seqs(cfg: PieceConfig):
    return np.random.SeedSequence(cfg.index).spawn(3)


def _lexicon(cfg: PieceConfig) -> List[Tuple[int, ...]]:
    rng = np.random.default_rng(_seqs(cfg)[0])
    p = 1.0 / np.arange(1, 27, dtype=np.float64)
    p = rng.permutation(p / p.sum())
    lens = rng.integers(3, 10, size=cfg.n_lexicon)
    words = {tuple(int(c) for c in rng.choice(26, size=int(L), p=p)) for L in lens}
    return sorted(words)


def _cased(piece: Tuple[int, ...], how: str) -> Tuple[int, ...]:
    out = list(piece)
    idx = [i for i, c in enumerate(out) if c < 26]
    if how == "title":
        idx = idx[:1]
    for i in idx:
        out[i] += 27
    return tuple(out)


def vocab(cfg: PieceConfig) -> List[Tuple[int, ...]]:
    """Token id -> character codes (V pieces; the blank V is not listed)."""
    rng = np.random.default_rng(_seqs(cfg)[0].spawn(1)[0])
    lex = _lexicon(cfg)
    cnt: Counter = Counter()
    for w in lex:
        for k in range(1, min(5, len(w)) + 1):
            cnt[(WORD,) + w[:k]] += 1
        for k in range(2, 7):
            for i in range(1, len(w) - k + 1):
                cnt[w[i:i + k]] += 1
    cands = sorted(cnt, key=lambda s: (-cnt[s], s))
    toks: List[Tuple[int, ...]] = [(c,) for c in range(N_CHARS)]
    seen = set(toks)
    for s in cands:
        if len(toks) >= cfg.V:
            break
        for piece, keep in ((s, True), (_cased(s, "title"), rng.random() < cfg.title_frac),
                            (_cased(s, "upper"), rng.random() < cfg.upper_frac)):
            if keep and piece not in seen and len(toks) < cfg.V:
                toks.append(piece)
                seen.add(piece)
    if len(toks) < cfg.V:
        raise ValueError("lexicon too small for the vocabulary size")
    return toks


def vocab_csr(toks: Sequence[Sequence[int]]):
    ptr = np.zeros(len(toks) + 1, dtype=np.int64)
    ptr[1:] = np.cumsum([len(t) for t in toks])
    chars = np.asarray([c for t in toks for c in t], dtype=np.int32)
    return ptr, chars


def phrases(cfg: PieceConfig, streams: Optional[Sequence[int]] = None) -> List[List[Tuple[int, ...]]]:
    """Per-stream phrase lists as character-code strings (random casing)."""
    if streams is None:
        streams = range(cfg.B)
    lex = _lexicon(cfg)
    r = np.arange(1, len(lex) + 1, dtype=np.float64) ** -1.0
    pw = r / r.sum()
    seq = _seqs(cfg)[1]
    out = []
    for b in streams:
        rng = np.random.default_rng(
            np.random.SeedSequence(entropy=seq.entropy, spawn_key=seq.spawn_key + (b,)))
        lst = []
        for _ in range(cfg.n_phrases):
            n = int(rng.integers(cfg.words_lo, cfg.words_hi + 1))
            ph: List[int] = []
            for wi in rng.choice(len(lex), size=n, p=pw):
                u = rng.random()
                how = "lower" if u < 0.7 else ("title" if u < 0.9 else "upper")
                word = (WORD,) + lex[int(wi)]
                ph.extend(word if how == "lower" else _cased(word, how))
            lst.append(tuple(ph))
        out.append(lst)
    return out


def phrase_csr(lists: Sequence[Sequence[Sequence[int]]]):
    mp, pp, chars = [0], [0], []
    for lst in lists:
        for ph in lst:
            chars.extend(ph)
            pp.append(pp[-1] + len(ph))
        mp.append(len(pp) - 1)
    return (np.asarray(mp, np.int64), np.asarray(pp, np.int64), np.asarray(chars, np.int32))


def spellings(toks: Sequence[Sequence[int]]) -> Dict[Tuple[int, ...], List[int]]:
    """Lowercased spelling -> the token ids spelled that way (any casing)."""
    out: Dict[Tuple[int, ...], List[int]] = {}
    for v, t in enumerate(toks):
        out.setdefault(tuple(int(LOWER[c]) for c in t), []).append(v)
    return out


def random_spelling(phrase: Sequence[int], spell: Dict[Tuple[int, ...], List[int]],
                    rng: np.random.Generator, longest: int = 7) -> List[int]:
    """Token ids spelling the phrase: a random piece at every position, then a
    random casing of that piece."""
    low = tuple(int(LOWER[c]) for c in phrase)
    out, i = [], 0
    while i < len(low):
        opts = [m for m in range(1, min(longest, len(low) - i) + 1) if low[i:i + m] in spell]
        m = opts[int(rng.integers(0, len(opts)))]
        ids = spell[low[i:i + m]]
        out.append(ids[int(rng.integers(0, len(ids)))])
        i += m
    return out


def plants(cfg: PieceConfig, b: int, toks=None, lst=None) -> List[Tuple[int, int]]:
    """(step, token) pairs boosted in stream b: one spelled phrase per 16 steps."""
    toks = vocab(cfg) if toks is None else toks
    lst = phrases(cfg, [b])[0] if lst is None else lst
    spell = spellings(toks)
    seq = _seqs(cfg)[2]
    rng = np.random.default_rng(
        np.random.SeedSequence(entropy=seq.entropy, spawn_key=seq.spawn_key + (b, 1)))
    out = []
    for s0 in range(0, cfg.T - 16 + 1, 16):
        sp = random_spelling(lst[int(rng.integers(0, len(lst)))], spell, rng)
        if len(sp) > 16:
            continue
        start = s0 + int(rng.integers(0, 16 - len(sp) + 1))
        out.extend((start + i, v) for i, v in enumerate(sp))
    return out


def _base(cfg: PieceConfig) -> Config:
    return Config(cfg.index, cfg.name, B=cfg.B, K=cfg.K, V=cfg.V, T=cfg.T, chunk=cfg.chunk,
                  dtype="f32", n_phrases=cfg.n_phrases, len_lo=1, len_hi=1,
                  token_dist="uniform", zipf_s=0.0, logit_std=cfg.logit_std,
                  blank_offset=cfg.blank_offset, n_case=1)


def logit_chunks(cfg: PieceConfig, chunk: int, t0: int = 0, t1: Optional[int] = None,
                 plant_map: Optional[dict] = None):
    """(ta, tb, rows [tb-ta, B, K, V+1]) slices: float32, or uint16 bf16 bits.
    ``plant_map`` (step -> [(stream, token)]) may be passed to avoid recomputing it."""
    from .synth import logit_chunks as base_chunks
    if t1 is None:
        t1 = cfg.T
    if plant_map is None:
        toks = vocab(cfg)
        plant_map = {}
        for b, lst in enumerate(phrases(cfg)):
            for t, v in plants(cfg, b, toks, lst):
                plant_map.setdefault(t, []).append((b, v))
    for ta, tb, rows in base_chunks(_base(cfg), chunk, t0, t1):
        for t in range(ta, tb):
            for b, v in plant_map.get(t, ()):
                rows[t - ta, b, :, v] += np.float32(cfg.plant_boost)
        if cfg.dtype == "f32":
            yield ta, tb, rows
        else:
            yield ta, tb, _f32_to_bf16_bits(rows)


def logits(cfg: PieceConfig, t0: int = 0, t1: Optional[int] = None) -> np.ndarray:
    if t1 is None:
        t1 = cfg.T
    out = np.empty((t1 - t0, cfg.B, cfg.K, cfg.Vp1),
                   dtype=np.float32 if cfg.dtype == "f32" else np.uint16)
    for ta, tb, rows in logit_chunks(cfg, 16, t0, t1):
        out[ta - t0:tb - t0] = rows
    return out
