"""Shared helpers of the GPU parity tests: run the HIP path, run the oracle."""

from __future__ import annotations

import os
import sys
import tempfile
import time
from typing import Dict, List, Optional, Sequence

import numpy as np

import oracle
import workloads as W


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def oracle_graphs(cfg, lists, streams, model_ids):
    cm = W.class_map(cfg)
    out = {}
    for b in streams:
        m = int(model_ids[b])
        if m >= 0 and m not in out:
            out[m] = oracle.build_graph(lists[m], cm, token_w=cfg.token_w,
                                        end_bonus=cfg.end_bonus)
    return out


def device_rows(cfg, streams, device="cuda", spill: Optional[str] = None):
    """Upload the full logits of cfg slice by slice; keep the sampled streams on the host.

    Returns (device tensor [T, B, K, V+1], host rows [T, S, K, V+1]). With
    ``spill`` (a file path) every row is also written to that file as a raw
    [T, B, K, V+1] array, for oracle worker processes to map."""
    import torch
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    hdt = np.float32 if cfg.dtype == "f32" else np.uint16
    dev = torch.empty((cfg.T, cfg.B, cfg.K, cfg.Vp1), dtype=dt, device=device)
    keep = np.empty((cfg.T, len(streams), cfg.K, cfg.Vp1), dtype=hdt)
    mm = None if spill is None else np.lib.format.open_memmap(
        spill, mode="w+", dtype=hdt, shape=(cfg.T, cfg.B, cfg.K, cfg.Vp1))
    sel = np.asarray(list(streams), dtype=np.int64)
    for ta, tb, rows in W.logit_chunks(cfg, 16):
        h = torch.from_numpy(rows if cfg.dtype == "f32" else rows.view(np.int16))
        dev[ta:tb].copy_(h.to(device).view(dt))
        keep[ta:tb] = rows[:, sel]
        if mm is not None:
            mm[ta:tb] = rows
    if mm is not None:
        mm.flush()
        del mm
    return dev, keep


def _oracle_part(args):
    """Worker (no GPU): the oracle on some streams of a named workload, with the
    logits read from a spilled [T, B, K, V+1] file."""
    name, streams, path = args
    cfg = W.config_by_name(name)
    cm = W.class_map(cfg)
    lists = W.phrases(cfg, streams)
    graphs = {i: oracle.build_graph(l, cm, token_w=cfg.token_w, end_bonus=cfg.end_bonus)
              for i, l in enumerate(lists)}
    mm = np.load(path, mmap_mode="r")
    rows = np.ascontiguousarray(mm[:, streams])
    del mm
    mids = list(range(len(streams)))
    if cfg.K == 1:
        return streams, oracle.greedy_decode(graphs, mids, rows, np.zeros(len(streams), np.int32))
    st, S = oracle.init_carry(mids, cfg.K)
    return streams, oracle.beam_decode(graphs, mids, rows, st, S)


def oracle_all_streams(cfg, path: str, parts: int = 64):
    """The oracle over every stream of a workload (stream b uses its own list,
    model b), in at most 16 GPU-free worker processes. Returns outputs shaped
    like greedy_decode's / beam_decode's for all B streams."""
    import multiprocessing as mp
    B = cfg.B
    chunks = [list(range(B))[i::parts] for i in range(min(parts, B))]
    procs = max(1, min(16, len(os.sched_getaffinity(0)), len(chunks)))
    greedy = cfg.K == 1
    shape = (cfg.T, B) if greedy else (cfg.T, B, cfg.K)
    if greedy:
        out = [np.zeros(shape, np.int32), np.zeros(shape, np.int32), np.zeros(shape, np.float32),
               np.zeros(B, np.int32)]
    else:
        out = [np.zeros(shape, np.int32), np.zeros(shape, np.int32), np.zeros(shape, np.int32),
               np.zeros(shape, np.float32), np.zeros(shape, np.float32)]
    t0 = time.time()
    done = 0
    with mp.get_context("spawn").Pool(procs) as pool:
        for streams, res in pool.imap_unordered(_oracle_part,
                                                [(cfg.name, c, path) for c in chunks]):
            for i in range(3 if greedy else 5):   # per-step outputs [T, B(, K)]
                out[i][:, streams] = res[i]
            if greedy:                              # the carry [B]
                out[3][streams] = res[3]
            done += 1
            if done % 8 == 0 or done == len(chunks):
                say(f"[oracle] {cfg.name}: {done}/{len(chunks)} parts, {time.time() - t0:.0f}s")
    return tuple(out)


def spill_path(tag: str) -> str:
    return os.path.join(tempfile.gettempdir(), f"tbias_rows_{tag}_{os.getpid()}.npy")


def gpu_greedy(dec, rows_dev, model_ids, chunk: int, states0=None):
    import torch
    T, B = rows_dev.shape[0], rows_dev.shape[1]
    mids, states, _ = dec.start(model_ids, 1)
    if states0 is not None:
        states.copy_(torch.as_tensor(states0, dtype=torch.int32, device=states.device))
    tok = torch.empty((T, B), dtype=torch.int32, device=rows_dev.device)
    st = torch.empty_like(tok)
    sc = torch.empty((T, B), dtype=torch.float32, device=rows_dev.device)
    for t0 in range(0, T, chunk):
        t1 = min(T, t0 + chunk)
        dec.greedy(rows_dev[t0:t1], mids, states, out=(tok[t0:t1], st[t0:t1], sc[t0:t1]))
    torch.cuda.synchronize()
    return tok.cpu().numpy(), st.cpu().numpy(), sc.cpu().numpy(), states.cpu().numpy()


def gpu_beam(dec, rows_dev, model_ids, chunk: int):
    import torch
    T, B, K = rows_dev.shape[0], rows_dev.shape[1], rows_dev.shape[2]
    mids, states, scores = dec.start(model_ids, K)
    i32 = dict(dtype=torch.int32, device=rows_dev.device)
    f32 = dict(dtype=torch.float32, device=rows_dev.device)
    outs = [torch.empty((T, B, K), **i32) for _ in range(3)] + \
           [torch.empty((T, B, K), **f32) for _ in range(2)]
    for t0 in range(0, T, chunk):
        t1 = min(T, t0 + chunk)
        dec.beam(rows_dev[t0:t1], mids, states, scores, out=tuple(o[t0:t1] for o in outs))
    torch.cuda.synchronize()
    return tuple(o.cpu().numpy() for o in outs) + (states.cpu().numpy(), scores.cpu().numpy())


def _score_error(a, b) -> float:
    """Largest |a - b| over the entries that differ (equal entries, infinite
    ones included, count 0; a NaN on either side counts as an error)."""
    if a.size == 0:
        return 0.0
    with np.errstate(invalid="ignore"):
        d = np.where(a == b, 0.0, np.abs(a.astype(np.float64) - b.astype(np.float64)))
    return float(np.nanmax(d)) if not np.isnan(d).any() else float("nan")


def compare_greedy(gpu, ref, streams, atol=1e-5, ref_streams=None):
    """gpu[i][:, streams] against ref[i][:, ref_streams] (default: the same columns)."""
    s = list(streams)
    r = s if ref_streams is None else list(ref_streams)
    tok, st, sc = (a[:, s] for a in gpu[:3])
    rtok, rst, rsc = (a[:, r] for a in ref[:3])
    bad = np.nonzero(tok != rtok)
    assert bad[0].size == 0, f"token mismatch at (t, stream-index) {list(zip(*bad))[:5]}"
    assert np.array_equal(st, rst), "state mismatch"
    err = _score_error(sc, rsc)
    assert err <= atol, f"score error {err}"
    return err


def compare_beam(gpu, ref, streams, atol=1e-5, ref_streams=None):
    s = list(streams)
    r = s if ref_streams is None else list(ref_streams)
    for i, n in enumerate(["tok", "parent", "state"]):
        bad = np.nonzero(gpu[i][:, s] != ref[i][:, r])
        assert bad[0].size == 0, f"{n} mismatch at {list(zip(*bad))[:5]}"
    assert np.array_equal(gpu[4][:, s], ref[4][:, r]), "accumulated score not bit-exact"
    err = _score_error(gpu[3][:, s], ref[3][:, r])
    assert err <= atol, f"step score error {err}"
    return err
