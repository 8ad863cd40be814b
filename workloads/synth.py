"""Synthetic workloads shaped like the paper's streaming, batched and beam decoding runs.

The paper evaluates on Contextual Earnings-22 and an internal medical set with
128 concurrent streams (Sec. III-B, Table III). Neither the audio, the models nor
a tokenizer are available, so every input here is synthetic and seeded:

* a vocabulary of V non-blank token ids plus one blank (id V), where the first
  3*n_case ids form 3-way case classes (lower / upper / title blocks, the
  case-insensitive setting of Sec. II-A) and the remaining ids are caseless;
* per-stream phrase lists given as token ids (Sec. II-B: every stream carries
  its own context list);
* joint-logit rows [T, B, K, V+1] standing in for the Transducer joint output.

Random streams: numpy ``default_rng`` over ``SeedSequence(seed)`` with
seed = the workload's index. Child 0 of that sequence drives the phrase lists
(one grandchild per stream, so a stream's list does not depend on B), child 1
the logits (one generator per time step, so any time slice can be regenerated
on its own).
"""

from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import List, Optional, Sequence, Tuple

import numpy as np


@dataclass(frozen=True)
class Config:
    index: int          # seed and workload index
    name: str
    B: int              # streams
    K: int              # hypotheses per stream (1 = greedy)
    V: int              # non-blank vocabulary size; blank id = V
    T: int              # decoding steps
    chunk: int          # steps per streaming call
    dtype: str          # "f32" or "bf16"
    n_phrases: int      # phrases per stream
    len_lo: int         # phrase length range (tokens, inclusive)
    len_hi: int
    token_dist: str     # "uniform" or "zipf"
    zipf_s: float
    logit_std: float
    blank_offset: float
    n_case: int         # number of 3-way case classes
    plant_frac: float = 0.0    # fraction of each list that is planted into the logits
    plant_boost: float = 0.0   # logit offset added at planted steps
    token_w: float = 1.0       # per-token boosting score w
    end_bonus: float = 2.0     # end-of-phrase bonus
    alpha: float = 1.0         # per-model boosting weight
    notes: str = ""

    @property
    def Vp1(self) -> int:
        return self.V + 1

    @property
    def rows(self) -> int:
        return self.T * self.B * self.K

    @property
    def itemsize(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def logit_bytes(self) -> int:
        return self.rows * self.Vp1 * self.itemsize


CONFIGS: Tuple[Config, ...] = (
    Config(0, "tiny", B=1, K=1, V=256, T=50, chunk=50, dtype="f32", n_phrases=10,
           len_lo=1, len_hi=4, token_dist="uniform", zipf_s=0.0, logit_std=1.0,
           blank_offset=0.0, n_case=64),
    Config(1, "batched", B=32, K=1, V=1024, T=500, chunk=500, dtype="f32",
           n_phrases=100, len_lo=1, len_hi=6, token_dist="zipf", zipf_s=1.2,
           logit_std=1.0, blank_offset=2.0, n_case=1024 // 9),
    Config(2, "streaming", B=128, K=1, V=1024, T=1024, chunk=16, dtype="f32",
           n_phrases=1000, len_lo=1, len_hi=10, token_dist="zipf", zipf_s=1.1,
           logit_std=1.0, blank_offset=1.5, n_case=1024 // 9),
    Config(3, "beam", B=64, K=8, V=1024, T=256, chunk=256, dtype="f32",
           n_phrases=1000, len_lo=1, len_hi=10, token_dist="zipf", zipf_s=1.1,
           logit_std=1.5, blank_offset=0.0, n_case=1024 // 9),
    Config(4, "stress_greedy", B=256, K=1, V=8192, T=256, chunk=256, dtype="bf16",
           n_phrases=10000, len_lo=1, len_hi=12, token_dist="zipf", zipf_s=1.0,
           logit_std=1.0, blank_offset=0.0, n_case=8192 // 12, plant_frac=0.1,
           plant_boost=4.0),
    Config(4, "stress_beam", B=256, K=4, V=8192, T=256, chunk=256, dtype="bf16",
           n_phrases=10000, len_lo=1, len_hi=12, token_dist="zipf", zipf_s=1.0,
           logit_std=1.0, blank_offset=0.0, n_case=8192 // 12, plant_frac=0.1,
           plant_boost=4.0),
)


def config_by_name(name: str, **overrides) -> Config:
    for c in CONFIGS:
        if c.name == name:
            return replace(c, **overrides) if overrides else c
    raise KeyError(name)


# ---------------------------------------------------------------------------
# vocabulary


def class_map(cfg: Config) -> np.ndarray:
    """Token -> case class. Class id = the lowercase member's token id.

    Ids [0, n) are lowercase, [n, 2n) their uppercase and [2n, 3n) their
    title-case variants; every other non-blank id is its own class. The blank
    (id V) maps to -1.
    """
    n, V = cfg.n_case, cfg.V
    if 3 * n > V:
        raise ValueError("case classes exceed the vocabulary")
    cm = np.arange(V + 1, dtype=np.int32)
    cm[n:2 * n] -= n
    cm[2 * n:3 * n] -= 2 * n
    cm[V] = -1
    return cm


def class_members(cfg: Config, tok: int) -> List[int]:
    """All token ids sharing tok's case class (ascending)."""
    n = cfg.n_case
    if tok < 3 * n:
        c = tok % n
        return [c, c + n, c + 2 * n]
    return [tok]


# ---------------------------------------------------------------------------
# phrase lists


def _graph_seq(cfg: Config) -> np.random.SeedSequence:
    return np.random.SeedSequence(cfg.index).spawn(2)[0]


def _logit_seq(cfg: Config) -> np.random.SeedSequence:
    return np.random.SeedSequence(cfg.index).spawn(2)[1]


def _stream_seqs(cfg: Config, b: int) -> Sequence[np.random.SeedSequence]:
    # Grandchild b of the graph child; its two children drive the phrase list
    # and the planting schedule of stream b. Spawning is deterministic, so the
    # result does not depend on how many streams are requested.
    g = _graph_seq(cfg)
    gc = np.random.SeedSequence(entropy=g.entropy, spawn_key=g.spawn_key + (b,))
    return gc.spawn(2)


def _token_probs(cfg: Config) -> Optional[np.ndarray]:
    if cfg.token_dist == "uniform":
        return None
    r = np.arange(1, cfg.V + 1, dtype=np.float64)  # rank r <-> token id r-1
    p = r ** (-cfg.zipf_s)
    return p / p.sum()


def phrases(cfg: Config, streams: Optional[Sequence[int]] = None) -> List[List[np.ndarray]]:
    """Per-stream phrase lists; each phrase is an int32 array of token ids in [0, V)."""
    if streams is None:
        streams = range(cfg.B)
    p = _token_probs(cfg)
    out = []
    for b in streams:
        rng = np.random.default_rng(_stream_seqs(cfg, b)[0])
        lens = rng.integers(cfg.len_lo, cfg.len_hi + 1, size=cfg.n_phrases)
        total = int(lens.sum())
        if p is None:
            toks = rng.integers(0, cfg.V, size=total)
        else:
            toks = rng.choice(cfg.V, size=total, p=p)
        toks = toks.astype(np.int32)
        out.append(np.split(toks, np.cumsum(lens)[:-1]))
    return out


def phrase_csr(lists: Sequence[Sequence[np.ndarray]]):
    """Flatten per-model phrase lists into (model_phrase_ptr, phrase_tok_ptr, tokens)."""
    mp = [0]
    tp = [0]
    toks: List[np.ndarray] = []
    for lst in lists:
        for ph in lst:
            toks.append(np.asarray(ph, dtype=np.int32))
            tp.append(tp[-1] + len(ph))
        mp.append(len(tp) - 1)
    tokens = np.concatenate(toks) if toks else np.zeros(0, np.int32)
    return (np.asarray(mp, np.int64), np.asarray(tp, np.int64), tokens.astype(np.int32))


def model_ids(cfg: Config) -> np.ndarray:
    """Stream b uses model b (its own list)."""
    return np.arange(cfg.B, dtype=np.int32)


# ---------------------------------------------------------------------------
# planted targets (stress workload)


def plants(cfg: Config, b: int, lst: Optional[Sequence[np.ndarray]] = None) -> List[Tuple[int, int]]:
    """(step, token) pairs whose logit gets +plant_boost in stream b.

    The first plant_frac of the stream's list are its targets (the list is
    i.i.d., so this is a random subset); the rest are distractors and are never
    planted. The T steps are cut into slots of 16; each slot holds at most one
    planted target occurrence (non-overlapping), spelled with a random case
    variant of each of its tokens.
    """
    if cfg.plant_frac <= 0.0:
        return []
    if lst is None:
        lst = phrases(cfg, [b])[0]
    n_t = max(1, int(round(cfg.plant_frac * len(lst))))
    rng = np.random.default_rng(_stream_seqs(cfg, b)[1])
    out = []
    slot = 16
    for s0 in range(0, cfg.T - slot + 1, slot):
        ph = lst[int(rng.integers(0, n_t))]
        L = len(ph)
        if L > slot:
            continue
        start = s0 + int(rng.integers(0, slot - L + 1))
        for i, tok in enumerate(ph):
            mem = class_members(cfg, int(tok))
            out.append((start + i, mem[int(rng.integers(0, len(mem)))]))
    return out


# ---------------------------------------------------------------------------
# logits


def _f32_to_bf16_bits(x: np.ndarray, out: Optional[np.ndarray] = None,
                      tmp: Optional[np.ndarray] = None) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest even), returned as uint16 bits.

    Finite inputs only (the generators never produce inf or nan). ``x`` is
    overwritten when ``tmp`` is given (scratch of the same shape, uint32)."""
    if tmp is None:
        u = np.array(x, dtype=np.float32, copy=True).view(np.uint32)
        lsb = np.right_shift(u, 16)
    else:
        u = x.view(np.uint32)
        lsb = np.right_shift(u, 16, out=tmp)
    np.bitwise_and(lsb, 1, out=lsb)
    u += np.uint32(0x7FFF)
    u += lsb
    np.right_shift(u, 16, out=u)
    if out is None:
        return u.astype(np.uint16)
    out[...] = u
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bits to float32."""
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _plant_map(cfg: Config, t0: int, t1: int) -> dict:
    out: dict = {}
    if cfg.plant_frac > 0.0:
        for b in range(cfg.B):
            for (t, tok) in plants(cfg, b):
                if t0 <= t < t1:
                    out.setdefault(t, []).append((b, tok))
    return out


def logit_chunks(cfg: Config, chunk: int, t0: int = 0, t1: Optional[int] = None):
    """Yield (ta, tb, rows) for consecutive time slices [ta, tb) of the logits.

    ``rows`` has shape [tb-ta, B, K, V+1] (float32, or uint16 bf16 bits) and is
    a buffer reused by the next slice: copy what must be kept. Each time step
    draws from its own generator (SFC64 over the step's SeedSequence), so the
    values never depend on the slicing.
    """
    if t1 is None:
        t1 = cfg.T
    seq = _logit_seq(cfg)
    B, K, Vp1 = cfg.B, cfg.K, cfg.Vp1
    pm = _plant_map(cfg, t0, t1)
    z = np.empty((B, K, Vp1), dtype=np.float32)
    tmp = np.empty((B, K, Vp1), dtype=np.uint32) if cfg.dtype == "bf16" else None
    buf = np.empty((min(chunk, max(1, t1 - t0)), B, K, Vp1),
                   dtype=np.float32 if cfg.dtype == "f32" else np.uint16)
    for ta in range(t0, t1, chunk):
        tb = min(t1, ta + chunk)
        for t in range(ta, tb):
            ts = np.random.SeedSequence(entropy=seq.entropy, spawn_key=seq.spawn_key + (t,))
            rng = np.random.Generator(np.random.SFC64(ts))
            zz = buf[t - ta] if cfg.dtype == "f32" else z
            rng.standard_normal(dtype=np.float32, out=zz)
            if cfg.logit_std != 1.0:
                zz *= np.float32(cfg.logit_std)
            if cfg.blank_offset != 0.0:
                zz[:, :, cfg.V] += np.float32(cfg.blank_offset)
            for (b, tok) in pm.get(t, ()):
                zz[b, :, tok] += np.float32(cfg.plant_boost)
            if cfg.dtype != "f32":
                _f32_to_bf16_bits(zz, out=buf[t - ta], tmp=tmp)
        yield ta, tb, buf[:tb - ta]


def logits(cfg: Config, t0: int = 0, t1: Optional[int] = None,
           streams: Optional[Sequence[int]] = None) -> np.ndarray:
    """Joint-logit rows [t1-t0, B', K, V+1]; float32, or uint16 bf16 bits for bf16.

    ``streams`` selects a subset of streams (rows are drawn for all B streams
    and then sliced, so values do not depend on the subset).
    """
    if t1 is None:
        t1 = cfg.T
    sel = None if streams is None else np.asarray(list(streams), dtype=np.int64)
    nb = cfg.B if sel is None else len(sel)
    out = np.empty((t1 - t0, nb, cfg.K, cfg.Vp1),
                   dtype=np.float32 if cfg.dtype == "f32" else np.uint16)
    for ta, tb, rows in logit_chunks(cfg, 16, t0, t1):
        out[ta - t0:tb - t0] = rows if sel is None else rows[:, sel]
    return out
