"""The greedy hand-off timeout path, forced from the host.

The waves of a segmented greedy workgroup pass exact states along the
segments through LDS, with a bounded wait. tb_debug_set_spin_limit(1) makes
that wait give up after one poll, so later waves write TB_STATE_TIMEOUT
instead of repairing; every kernel still ends normally. Checked: every row is
either marked TB_STATE_TIMEOUT or equal to the oracle, the carry of a stream
with unrepaired rows is TB_STATE_TIMEOUT, and a carried TB_STATE_TIMEOUT is
sticky (the next call decodes that stream without biasing and writes
TB_STATE_TIMEOUT again) until the stream is reset.
"""

import numpy as np
import pytest

import oracle
import workloads as W
from paper_2608_21343_amd import capi
from tests.gpu_cases import gpu_greedy, oracle_graphs, say

pytestmark = pytest.mark.gpu


@pytest.fixture
def tiny_spin_limit():
    capi.tb_debug_set_spin_limit(1)
    yield
    capi.tb_debug_set_spin_limit(0)


def _case():
    cfg = W.Config(400, "timeout", B=5, K=1, V=300, T=700, chunk=700, dtype="f32",
                   n_phrases=60, len_lo=1, len_hi=6, token_dist="zipf", zipf_s=1.2,
                   logit_std=1.0, blank_offset=1.0, n_case=40)
    return cfg, W.phrases(cfg), W.logits(cfg)


def test_forced_timeout_marks_rows_and_carry(tiny_spin_limit):
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg, lists, rows = _case()
    mids = W.model_ids(cfg)
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    say("[timeout] one long call with a hand-off wait of one poll")
    tok, st, sc, carry = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, cfg.T)
    graphs = oracle_graphs(cfg, lists, range(cfg.B), mids)
    ref = oracle.greedy_decode(graphs, mids, rows, np.zeros(cfg.B, np.int32))
    marked = st == capi.TB_STATE_TIMEOUT
    say(f"[timeout] rows marked: {int(marked.sum())} of {marked.size}")
    assert marked.any(), "a one-poll hand-off wait never gave up"
    ok = ~marked
    assert np.array_equal(tok[ok], ref[0][ok]) and np.array_equal(st[ok], ref[1][ok])
    assert np.max(np.abs(sc[ok] - ref[2][ok])) <= 1e-5
    for b in range(cfg.B):
        assert carry[b] in (capi.TB_STATE_TIMEOUT, ref[3][b])
        if marked[-1, b]:
            assert carry[b] == capi.TB_STATE_TIMEOUT


@pytest.mark.parametrize("chunk", [16, 700])
def test_carried_timeout_state_is_sticky_until_reset(chunk):
    import torch
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg, lists, rows = _case()
    mids = W.model_ids(cfg)
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    dev = to_device_logits(rows[:, :, 0, :])
    s0 = np.zeros(cfg.B, np.int32)
    s0[2] = capi.TB_STATE_TIMEOUT
    say(f"[timeout] carried TB_STATE_TIMEOUT, chunk {chunk}")
    tok, st, sc, carry = gpu_greedy(dec, dev, mids, chunk, states0=s0)
    assert np.all(st[:, 2] == capi.TB_STATE_TIMEOUT) and carry[2] == capi.TB_STATE_TIMEOUT
    z = rows[:, 2, 0, :]
    assert np.array_equal(tok[:, 2], np.argmax(z, axis=1))      # decoded without biasing
    graphs = oracle_graphs(cfg, lists, range(cfg.B), mids)
    others = [0, 1, 3, 4]
    ref = oracle.greedy_decode(graphs, mids, rows, np.zeros(cfg.B, np.int32), streams=others)
    assert np.array_equal(tok[:, others], ref[0][:, others])
    assert np.array_equal(st[:, others], ref[1][:, others])
    # the beam step keeps it sticky too
    K = 3
    m, bst, bsc = dec.start(mids, K)
    bst[2 * K] = capi.TB_STATE_TIMEOUT
    out = dec.beam(to_device_logits(np.repeat(rows[:64], K, axis=2)), m, bst, bsc)
    torch.cuda.synchronize()
    assert np.all(out[2].cpu().numpy()[:, 2] == capi.TB_STATE_TIMEOUT)
    # a reset restarts the stream
    m, gst, _ = dec.start(mids)
    gst[2] = capi.TB_STATE_TIMEOUT
    capi.tb_reset_stream(dec.arena, 2, int(mids[2]), 1, m, gst)
    torch.cuda.synchronize()
    assert int(gst[2].item()) == 0
