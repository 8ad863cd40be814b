"""Step calls from two host threads at once, each thread on its own HIP
stream, on one arena: every call's outputs equal those of the same calls made
one after another. The arena is only read by step calls, and the library's
host-side state (kernel choice, error messages) is safe to share between
threads."""

import threading

import numpy as np
import pytest

import workloads as W
from tests.gpu_cases import say

pytestmark = pytest.mark.gpu


def _case():
    cfg = W.Config(300, "threads", B=16, K=4, V=1024, T=96, chunk=96, dtype="f32",
                   n_phrases=200, len_lo=1, len_hi=8, token_dist="zipf", zipf_s=1.1,
                   logit_std=1.0, blank_offset=1.0, n_case=113)
    return cfg, W.phrases(cfg), W.logits(cfg)


def _greedy_loop(dec, rows_dev, mids, chunk):
    import torch
    T, B = rows_dev.shape[0], rows_dev.shape[1]
    m, st, _ = dec.start(mids)
    tok = torch.empty((T, B), dtype=torch.int32, device="cuda")
    sst = torch.empty_like(tok)
    sc = torch.empty((T, B), dtype=torch.float32, device="cuda")
    for t0 in range(0, T, chunk):
        dec.greedy(rows_dev[t0:t0 + chunk], m, st, out=(tok[t0:t0 + chunk], sst[t0:t0 + chunk],
                                                         sc[t0:t0 + chunk]))
    return tok, sst, sc, st


def _beam_loop(dec, rows_dev, mids, chunk):
    import torch
    T, B, K = rows_dev.shape[0], rows_dev.shape[1], rows_dev.shape[2]
    m, st, sc = dec.start(mids, K)
    outs = [torch.empty((T, B, K), dtype=torch.int32, device="cuda") for _ in range(3)] + \
           [torch.empty((T, B, K), dtype=torch.float32, device="cuda") for _ in range(2)]
    for t0 in range(0, T, chunk):
        dec.beam(rows_dev[t0:t0 + chunk], m, st, sc, out=tuple(o[t0:t0 + chunk] for o in outs))
    return tuple(outs) + (st, sc)


def _host(ts):
    return [t.cpu().numpy() for t in ts]


def test_two_threads_two_streams_one_arena():
    import torch
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg, lists, rows = _case()
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.arange(cfg.B, dtype=np.int32)
    mids[3] = -1
    beam_rows = to_device_logits(rows)
    greedy_rows = to_device_logits(np.ascontiguousarray(rows[:, :, 1, :]))
    torch.cuda.synchronize()
    jobs = [("greedy 16", lambda: _greedy_loop(dec, greedy_rows, mids, 16)),
            ("greedy 96", lambda: _greedy_loop(dec, greedy_rows, mids, 96)),
            ("beam 16", lambda: _beam_loop(dec, beam_rows, mids, 16)),
            ("beam 48", lambda: _beam_loop(dec, beam_rows, mids, 48))]
    want = {}
    for name, fn in jobs:
        want[name] = _host(fn())
        torch.cuda.synchronize()

    def worker(name, fn, stream, got, errors):
        try:
            with torch.cuda.stream(stream):
                for _ in range(3):
                    res = fn()
                    stream.synchronize()
                    got.append(_host(res))
        except Exception as e:  # re-raised below
            errors.append((name, e))

    for a, b in [(0, 1), (2, 3), (0, 2), (1, 3)]:
        say(f"[threads] {jobs[a][0]} beside {jobs[b][0]}")
        streams = [torch.cuda.Stream(), torch.cuda.Stream()]
        got = [[], []]
        errors = []
        th = [threading.Thread(target=worker, args=(jobs[j][0], jobs[j][1], streams[i], got[i],
                                                    errors))
              for i, j in enumerate((a, b))]
        for t in th:
            t.start()
        for t in th:
            t.join()
        assert not errors, errors
        for i, j in enumerate((a, b)):
            assert len(got[i]) == 3
            for rep in got[i]:
                for x, y in zip(rep, want[jobs[j][0]]):
                    assert np.array_equal(x, y), jobs[j][0]
