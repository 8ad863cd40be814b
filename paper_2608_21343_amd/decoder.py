"""Convenience wrapper: compile per-stream lists once, then step chunks.

Marshalling only (device buffers come from torch, all work runs in
libtbias.so). Mirrors the streaming use of Sec. II-C: states (and beam
scores) live on the device between calls, so a stream can be decoded chunk by
chunk.
"""

from __future__ import annotations

from typing import Optional, Sequence

import numpy as np
import torch

from . import capi


def to_device_logits(rows: np.ndarray, device="cuda") -> torch.Tensor:
    """float32 rows as float32; uint16 bfloat16 bits as bfloat16."""
    if rows.dtype == np.float32:
        return torch.from_numpy(np.ascontiguousarray(rows)).to(device)
    if rows.dtype == np.uint16:
        t = torch.from_numpy(np.ascontiguousarray(rows).view(np.int16)).to(device)
        return t.view(torch.bfloat16)
    raise TypeError(rows.dtype)


class BoostDecoder:
    def __init__(self, lists: Sequence[Sequence[np.ndarray]], class_map: np.ndarray,
                 token_w=1.0, end_bonus=2.0, scale=None, semantics: int = capi.TB_COMMIT,
                 device="cuda"):
        mp, tp, tk = _csr(lists)
        self.graphs = capi.tb_compile_graphs(mp, tp, tk, token_w, end_bonus, class_map,
                                             scale=scale, semantics=semantics)
        self.arena = capi.tb_graphs_upload(self.graphs, device=device)
        self.device = device
        self.V1 = int(len(class_map))

    @classmethod
    def variative(cls, lists, pieces, lower, tau: float, token_w=1.0, end_bonus=2.0,
                  scale=None, semantics: int = capi.TB_COMMIT, device="cuda") -> "BoostDecoder":
        """Phrase lists written in characters, compiled into variative BPE
        graphs over the piece vocabulary ``pieces`` (token id -> character
        codes) with lowercasing map ``lower``."""
        mp, pp, pc = [0], [0], []
        for lst in lists:
            for ph in lst:
                pc.extend(int(c) for c in ph)
                pp.append(pp[-1] + len(ph))
            mp.append(len(pp) - 1)
        tp = np.zeros(len(pieces) + 1, np.int64)
        tp[1:] = np.cumsum([len(t) for t in pieces])
        tc = np.asarray([c for t in pieces for c in t], np.int32)
        self = cls.__new__(cls)
        self.graphs = capi.tb_compile_variative(np.asarray(mp, np.int64), np.asarray(pp, np.int64),
                                                np.asarray(pc, np.int32), token_w, end_bonus, tp,
                                                tc, lower, tau, scale=scale, semantics=semantics)
        self.arena = capi.tb_graphs_upload(self.graphs, device=device)
        self.device = device
        self.V1 = len(pieces) + 1
        return self

    @classmethod
    def for_arena(cls, arena, device="cuda") -> "BoostDecoder":
        """A decoder over an existing device arena (for example a registry's)."""
        self = cls.__new__(cls)
        self.graphs = None
        self.arena = arena
        self.device = device
        self.V1 = int(arena.layout.v_plus_blank)
        return self

    def start(self, model_ids: Sequence[int], K: int = 1):
        """Device carry for len(model_ids) streams: (model_ids, states, scores)."""
        B = len(model_ids)
        mids = torch.tensor(np.asarray(model_ids, np.int32), device=self.device)
        states = torch.empty(B * K, dtype=torch.int32, device=self.device)
        scores = torch.empty(B * K, dtype=torch.float32, device=self.device)
        capi.tb_init_states(self.arena, B, K, mids, states, scores)
        return mids, states, scores

    def greedy(self, logits: torch.Tensor, mids, states, out=None):
        T, B = logits.shape[0], logits.shape[1]
        if out is None:
            out = (torch.empty((T, B), dtype=torch.int32, device=self.device),
                   torch.empty((T, B), dtype=torch.int32, device=self.device),
                   torch.empty((T, B), dtype=torch.float32, device=self.device))
        capi.tb_boost_step_greedy(self.arena, logits, mids, states, *out)
        return out

    def beam(self, logits: torch.Tensor, mids, states, scores, out=None):
        T, B, K = logits.shape[0], logits.shape[1], logits.shape[2]
        if out is None:
            i32 = dict(dtype=torch.int32, device=self.device)
            f32 = dict(dtype=torch.float32, device=self.device)
            out = (torch.empty((T, B, K), **i32), torch.empty((T, B, K), **i32),
                   torch.empty((T, B, K), **i32), torch.empty((T, B, K), **f32),
                   torch.empty((T, B, K), **f32))
        capi.tb_boost_step_beam(self.arena, logits, mids, states, scores, *out)
        return out

    def start_beam_stream(self, model_ids: Sequence[int], K: int, tree_cap: int):
        """Device carry of the streaming beam: a BeamCarry."""
        B = len(model_ids)
        dev = self.device
        c = BeamCarry(
            mids=torch.tensor(np.asarray(model_ids, np.int32), device=dev),
            states=torch.empty(B * K, dtype=torch.int32, device=dev),
            scores=torch.empty(B * K, dtype=torch.float32, device=dev),
            hyps=torch.empty((B * K, capi.HYP_WORDS), dtype=torch.int64, device=dev),
            tree=(torch.zeros((B, tree_cap, 2), dtype=torch.int32, device=dev)
                  if tree_cap > 0 else None),
            tree_len=torch.empty(B, dtype=torch.int32, device=dev))
        capi.tb_init_beam_stream(self.arena, B, K, c.mids, c.states, c.scores, c.hyps,
                                 c.tree_len)
        return c

    def beam_stream(self, logits: torch.Tensor, carry: "BeamCarry", recombine: bool = True,
                    out=None):
        T, B, K = logits.shape[0], logits.shape[1], logits.shape[2]
        if out is None:
            i32 = dict(dtype=torch.int32, device=self.device)
            f32 = dict(dtype=torch.float32, device=self.device)
            out = (torch.empty((T, B, K), **i32), torch.empty((T, B, K), **i32),
                   torch.empty((T, B, K), **i32), torch.empty((T, B, K), **f32),
                   torch.empty((T, B, K), **f32))
        capi.tb_boost_step_beam_stream(self.arena, logits, carry.mids, carry.states, carry.scores,
                                       carry.hyps, carry.tree, carry.tree_len, *out,
                                       recombine=recombine)
        return out


class BeamCarry:
    """Device state of streaming beams: model ids [B], states and scores
    [B*K], tb_hyp records [B*K, 3] (int64 words), trees [B, cap, 2], tree
    lengths [B]."""

    def __init__(self, mids, states, scores, hyps, tree, tree_len):
        self.mids, self.states, self.scores = mids, states, scores
        self.hyps, self.tree, self.tree_len = hyps, tree, tree_len


def _csr(lists):
    mp = [0]
    tp = [0]
    toks = []
    for lst in lists:
        for ph in lst:
            toks.append(np.asarray(ph, dtype=np.int32))
            tp.append(tp[-1] + len(ph))
        mp.append(len(tp) - 1)
    tk = np.concatenate(toks).astype(np.int32) if toks else np.zeros(0, np.int32)
    return np.asarray(mp, np.int64), np.asarray(tp, np.int64), tk
