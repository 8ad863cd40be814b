"""Vocabularies at both ends of what the boundary accepts, one token plus the
blank (V+1 = 2) and V+1 = 32768, through the greedy and beam step calls,
against the oracle. The dispatch picks the kernels; at V+1 = 32768 these are
the reference kernels, whose per-class override table must fit the LDS.

Phrases are planted in the logits, so the biased moves are taken; a stream
on model -1 and one on an empty list ride along."""

import numpy as np
import pytest

import oracle
from paper_2608_21343_amd import capi
from tests.gpu_cases import compare_beam, compare_greedy, gpu_beam, gpu_greedy, say
from workloads.synth import _f32_to_bf16_bits

pytestmark = pytest.mark.gpu

ATOL = 1e-5


def _rows(V, lists, mids, T, K, seed, plant, dtype):
    rng = np.random.default_rng(seed)
    B = len(mids)
    rows = rng.normal(0, 1, (T, B, K, V + 1)).astype(np.float32)
    rows[..., V] += np.float32(1.0)
    for b, m in enumerate(mids):
        if m < 0 or not lists[m]:
            continue
        t = 1
        while True:
            ph = lists[m][int(rng.integers(len(lists[m])))]
            if t + len(ph) > T:
                break
            for i, v in enumerate(ph):
                rows[t + i, b, :, int(v)] += np.float32(plant)
            t += len(ph) + int(rng.integers(1, 4))
    return np.ascontiguousarray(_f32_to_bf16_bits(rows) if dtype == "bf16" else rows)


def _run(V, cm, lists, mids, T, K, seed, plant, dtype, chunk):
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    mids = np.asarray(mids, np.int32)
    rows = _rows(V, lists, mids, T, K, seed, plant, dtype)
    dec = BoostDecoder([[np.asarray(p, np.int32) for p in l] for l in lists], cm,
                       token_w=1.0, end_bonus=2.0)
    graphs = {int(m): oracle.build_graph(lists[m], cm, token_w=1.0, end_bonus=2.0)
              for m in set(mids.tolist()) if m >= 0}
    if K == 1:
        gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, chunk)
        st0 = np.where(mids >= 0, 0, -1).astype(np.int32)
        ref = oracle.greedy_decode(graphs, mids, rows[:, :, 0, :], st0)
        compare_greedy(gpu, ref, range(len(mids)), ATOL)
        states = gpu[1]
    else:
        gpu = gpu_beam(dec, to_device_logits(rows), mids, chunk)
        st0, S0 = oracle.init_carry(mids, K)
        ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
        compare_beam(gpu, ref, range(len(mids)), ATOL)
        states = gpu[2]
    # the planted phrases were followed: some stream left the root
    assert np.any(states[:, [b for b, m in enumerate(mids) if m >= 0]] > 0)


@pytest.mark.parametrize("K,dtype", [(1, "f32"), (1, "bf16"), (2, "f32")])
def test_one_token_vocabulary(K, dtype):
    cm = np.array([0, -1], np.int32)
    lists = [[[0]], [[0, 0, 0], [0, 0]], []]
    say(f"[extremes] V+1 = 2 K={K} {dtype}")
    _run(1, cm, lists, [0, 1, 2, -1], T=40, K=K, seed=1, plant=3.0, dtype=dtype, chunk=16)


def _largest():
    V = 32767
    n_case = 2000
    cm = np.arange(V + 1, dtype=np.int32)
    cm[n_case:2 * n_case] -= n_case
    cm[2 * n_case:3 * n_case] -= 2 * n_case
    cm[V] = -1
    rng = np.random.default_rng(7)
    lists = []
    for m in range(3):
        lst = [[int(t) for t in rng.integers(0, V, size=int(rng.integers(1, 7)))]
               for _ in range(40)]
        lst.append([V - 1, 0, V - 1])  # the largest token id, a case class member
        lst.append([n_case + 5, 2 * n_case + 5, 5])
        lists.append(lst)
    lists.append([])
    return V, cm, lists


@pytest.mark.parametrize("K,dtype,chunk", [(1, "f32", 24), (1, "bf16", 7), (2, "f32", 24),
                                           (3, "bf16", 10)])
def test_largest_vocabulary(K, dtype, chunk):
    V, cm, lists = _largest()
    say(f"[extremes] V+1 = {V + 1} K={K} {dtype} chunk={chunk}")
    _run(V, cm, lists, [0, 1, 2, 3, -1], T=24, K=K, seed=3, plant=5.0, dtype=dtype, chunk=chunk)


def test_largest_vocabulary_is_the_limit():
    cm = np.zeros(32770, np.int32)
    cm[-1] = -1
    with pytest.raises(capi.TbError) as e:
        capi.tb_compile_graphs([0, 1], [0, 1], [0], 1.0, 2.0, cm)
    assert e.value.code == capi.TB_ERANGE


def test_largest_vocabulary_streaming_beam():
    """The streaming beam (recombination and tree) at V+1 = 32768: the
    reference kernel's stage, chunk by chunk against the oracle's."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    V, cm, lists = _largest()
    mids = np.asarray([0, 1, 2, 3, -1], np.int32)
    K, T = 3, 20
    rows = _rows(V, lists, mids, T, K, seed=5, plant=5.0, dtype="f32")
    dec = BoostDecoder([[np.asarray(p, np.int32) for p in l] for l in lists], cm,
                       token_w=1.0, end_bonus=2.0)
    graphs = {m: oracle.build_graph(lists[m], cm, token_w=1.0, end_bonus=2.0) for m in range(4)}
    say(f"[extremes] V+1 = {V + 1} streaming beam K={K}")
    rows_dev = to_device_logits(rows)
    carry = dec.start_beam_stream(mids, K, 256)
    ref = oracle.init_stream_carry(mids, K)
    for t0 in range(0, T, 8):
        gpu = [o.cpu().numpy() for o in dec.beam_stream(rows_dev[t0:t0 + 8], carry)]
        want = oracle.beam_decode_stream(graphs, mids, rows[t0:t0 + 8], ref, tree_cap=256)
        compare_beam(gpu, want, range(len(mids)), ATOL)
    assert np.array_equal(carry.states.cpu().numpy().reshape(len(mids), K), ref["states"])
