"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Every workload runs at its full size on the device, in the launch pattern the
benchmark uses (streaming chunks of 16 for the streaming workload, one call
per workload otherwise), and the oracle recomputes every stream (in at most 16
worker processes). Bar: selected tokens, graph states and beam parents
bit-exact; accumulated beam scores bit-exact; per-step fused scores within
1e-5 absolute.
"""

import os

import numpy as np
import pytest

import oracle
import workloads as W
from paper_2608_21343_amd import capi
from tests.gpu_cases import (compare_beam, compare_greedy, device_rows, gpu_beam,
                             gpu_greedy, oracle_all_streams, oracle_graphs, say, spill_path)

pytestmark = pytest.mark.gpu

ATOL = 1e-5


def _decoder(cfg, lists):
    from paper_2608_21343_amd.decoder import BoostDecoder
    return BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)


def _full_size(name, run):
    """Full workload on the device in its launch pattern, the oracle on every stream."""
    cfg = W.config_by_name(name)
    say(f"[parity] {name}: generating B={cfg.B} K={cfg.K} T={cfg.T} V+1={cfg.Vp1} {cfg.dtype}")
    lists = W.phrases(cfg)
    dec = _decoder(cfg, lists)
    mids = W.model_ids(cfg)
    path = spill_path(name)
    try:
        dev, _ = device_rows(cfg, [], spill=path)
        say(f"[parity] {name}: running HIP path, chunk={cfg.chunk}")
        gpu = run(dec, dev, mids, cfg.chunk)
        del dev
        say(f"[parity] {name}: oracle on all {cfg.B} streams")
        ref = oracle_all_streams(cfg, path)
    finally:
        if os.path.exists(path):
            os.remove(path)
    return cfg, gpu, ref


@pytest.mark.parametrize("name", ["tiny", "batched", "streaming", "stress_greedy"])
def test_greedy_full_size(name):
    cfg, gpu, ref = _full_size(name, lambda dec, dev, mids, ch: gpu_greedy(dec, dev[:, :, 0, :],
                                                                          mids, ch))
    err = compare_greedy(gpu, ref, range(cfg.B), ATOL)
    assert np.array_equal(gpu[3], ref[3]), "carried states differ"
    say(f"[parity] greedy {name}: ok on all {cfg.B} streams, max score error {err:.2e}")


@pytest.mark.parametrize("name", ["beam", "stress_beam"])
def test_beam_full_size(name):
    cfg, gpu, ref = _full_size(name, gpu_beam)
    err = compare_beam(gpu, ref, range(cfg.B), ATOL)
    say(f"[parity] beam {name}: ok on all {cfg.B} streams, max step score error {err:.2e}")


def _small_case(seed=0, B=6, V=200, n_case=20, T=64, K=1, dtype="f32"):
    cfg = W.Config(100 + seed, "small", B=B, K=K, V=V, T=T, chunk=T, dtype=dtype,
                   n_phrases=40, len_lo=1, len_hi=5, token_dist="zipf", zipf_s=1.1,
                   logit_std=1.0, blank_offset=1.0, n_case=n_case)
    return cfg, W.phrases(cfg), W.logits(cfg)


def test_greedy_chunk_invariance():
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg = W.config_by_name("streaming")
    lists = W.phrases(cfg)
    rows = W.logits(cfg, 0, 96)
    dec = _decoder(cfg, lists)
    mids = W.model_ids(cfg)
    dev = to_device_logits(rows[:, :, 0, :])
    ref = gpu_greedy(dec, dev, mids, 96)
    for ch in (1, 7, 16):
        out = gpu_greedy(dec, dev, mids, ch)
        for a, b in zip(ref, out):
            assert np.array_equal(a, b), f"chunk {ch} differs"
    again = gpu_greedy(dec, dev, mids, 96)
    for a, b in zip(ref, again):
        assert np.array_equal(a, b), "not deterministic"


def test_beam_chunk_invariance():
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg, lists, rows = _small_case(1, K=4, T=40)
    dec = _decoder(cfg, lists)
    mids = W.model_ids(cfg)
    dev = to_device_logits(rows)
    ref = gpu_beam(dec, dev, mids, 40)
    for ch in (1, 7, 16):
        out = gpu_beam(dec, dev, mids, ch)
        for a, b in zip(ref, out):
            assert np.array_equal(a, b), f"chunk {ch} differs"
    st0, S0 = oracle.init_carry(mids, cfg.K)
    graphs = oracle_graphs(cfg, lists, range(cfg.B), mids)
    o = oracle.beam_decode(graphs, mids, rows, st0, S0)
    compare_beam(ref, o, range(cfg.B), ATOL)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_mixed_model_ids_and_edge_streams(dtype):
    """Model -1, an empty list, an out-of-range id and ragged V+1 in one batch."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg, lists, rows = _small_case(2, B=7, V=300, dtype=dtype)   # V+1 = 301: ragged
    lists = list(lists[:5]) + [[]]                               # model 5: empty list
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.array([0, -1, 5, 3, 99, 4, 1], np.int32)            # 99: out of range
    dev = to_device_logits(rows[:, :, 0, :])
    gpu = gpu_greedy(dec, dev, mids, 17)
    ok = [0, 1, 2, 3, 5, 6]
    graphs = oracle_graphs(cfg, lists, ok, mids)
    st0 = np.array([0, -1, 0, 0, 0, 0, 0], np.int32)
    ref = oracle.greedy_decode(graphs, mids, rows, st0, streams=ok)
    compare_greedy(gpu, ref, ok, ATOL)
    assert np.all(gpu[1][:, 1] == -1)
    assert np.all(gpu[1][:, 2] == 0)                             # root-only graph
    assert np.all(gpu[1][:, 4] == -2)                            # invalid id: no biasing
    z = oracle.widen(rows[:, 4, 0, :])
    assert np.array_equal(gpu[0][:, 4], np.argmax(z, axis=1))


def test_padded_row_stride_and_T0():
    import torch
    from paper_2608_21343_amd import capi
    cfg, lists, rows = _small_case(3, B=5, V=255)
    dec = _decoder(cfg, lists)
    mids = W.model_ids(cfg)
    T, B, V1 = cfg.T, cfg.B, cfg.Vp1
    pad = torch.full((T, B, V1 + 7), 1e30, dtype=torch.float32, device="cuda")
    pad[:, :, :V1] = torch.from_numpy(rows[:, :, 0, :]).cuda()
    m, st, _ = dec.start(mids)
    tok = torch.empty((T, B), dtype=torch.int32, device="cuda")
    sst = torch.empty_like(tok)
    sc = torch.empty((T, B), dtype=torch.float32, device="cuda")
    capi.tb_boost_step_greedy(dec.arena, pad[:, :, :V1], m, st, tok, sst, sc, row_stride=V1 + 7)
    torch.cuda.synchronize()
    graphs = oracle_graphs(cfg, lists, range(B), mids)
    ref = oracle.greedy_decode(graphs, mids, rows, np.zeros(B, np.int32))
    compare_greedy((tok.cpu().numpy(), sst.cpu().numpy(), sc.cpu().numpy()), ref, range(B), ATOL)
    before = st.clone()
    capi.tb_boost_step_greedy(dec.arena, pad[:0, :, :V1], m, st, tok, sst, sc, T=0,
                              row_stride=V1 + 7)
    torch.cuda.synchronize()
    assert torch.equal(before, st)


def test_reset_stream_touches_only_that_stream():
    import torch
    from paper_2608_21343_amd import capi
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg, lists, rows = _small_case(4, B=4, K=3, T=30)
    dec = _decoder(cfg, lists)
    mids = W.model_ids(cfg)
    dev = to_device_logits(rows)
    m, st, sc = dec.start(mids, cfg.K)
    dec.beam(dev[:10], m, st, sc)
    torch.cuda.synchronize()
    st_before, sc_before = st.cpu().numpy().copy(), sc.cpu().numpy().copy()
    capi.tb_reset_stream(dec.arena, 2, -1, cfg.K, m, st, sc)
    torch.cuda.synchronize()
    st_a, sc_a, m_a = st.cpu().numpy(), sc.cpu().numpy(), m.cpu().numpy()
    K = cfg.K
    keep = [i for i in range(cfg.B * K) if i // K != 2]
    assert np.array_equal(st_a[keep], st_before[keep]) and np.array_equal(sc_a[keep], sc_before[keep])
    assert list(st_a[2 * K:3 * K]) == [-1] * K and m_a[2] == -1
    assert sc_a[2 * K] == 0 and np.all(np.isneginf(sc_a[2 * K + 1:3 * K]))
    # continuing after the reset equals a fresh run of that stream without a model
    o = dec.beam(dev[10:], m, st, sc)
    torch.cuda.synchronize()
    st0, S0 = oracle.init_carry([-1], K)
    ref = oracle.beam_decode({}, [-1], rows[10:, 2:3], st0, S0)
    assert np.array_equal(o[0].cpu().numpy()[:, 2], ref[0][:, 0])
    assert np.array_equal(o[4].cpu().numpy()[:, 2], ref[4][:, 0])


def test_stream_permutation_permutes_outputs():
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg, lists, rows = _small_case(5, B=8, T=48)
    dec = _decoder(cfg, lists)
    mids = W.model_ids(cfg)
    ref = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, 48)
    perm = np.array([3, 7, 0, 5, 1, 6, 2, 4])
    out = gpu_greedy(dec, to_device_logits(np.ascontiguousarray(rows[:, perm, 0, :])),
                     mids[perm], 48)
    for a, b in zip(ref[:3], out[:3]):
        assert np.array_equal(a[:, perm], b)


@pytest.mark.parametrize("name,T,chunk", [("tiny", 50, 50), ("batched", 500, 500),
                                          ("streaming", 1024, 1024), ("streaming", 200, 37),
                                          ("streaming", 96, 16), ("batched", 40, 7)])
def test_greedy_kernels_agree_with_reference_kernel(name, T, chunk):
    """The segmented and short-call kernels give the reference kernel's outputs:
    tokens, states and carries identical, scores within rounding of the
    normaliser. Whole-length calls make the segmented kernel split streams
    over several workgroups and run its boundary fix-up; calls of at most 16
    steps take the short-call kernel."""
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg = W.config_by_name(name)
    lists = W.phrases(cfg)
    rows = W.logits(cfg, 0, T)
    dec = _decoder(cfg, lists)
    mids = W.model_ids(cfg).copy()
    if cfg.B > 4:
        mids[1] = -1
    dev = to_device_logits(rows[:, :, 0, :])
    del rows
    say(f"[agree] seg vs ref: {name} T={T} chunk={chunk}")
    out = gpu_greedy(dec, dev, mids, chunk)
    with capi.kernels(greedy=capi.GREEDY_REF):
        ref = gpu_greedy(dec, dev, mids, chunk)
    bad = np.nonzero(out[0] != ref[0])
    assert bad[0].size == 0, f"token mismatch at (t, b) {list(zip(*bad))[:5]}"
    assert np.array_equal(out[1], ref[1]) and np.array_equal(out[3], ref[3])
    assert np.max(np.abs(out[2] - ref[2])) <= 2e-6


def _phrase_following_rows(rng, T, B, V, plen, blank_every=9, margin=3.0):
    """Logits whose boosted greedy path walks through the phrase 1..plen over
    and over (a blank every blank_every rows), each stream out of phase."""
    rows = rng.normal(0.0, 0.1, size=(T, B, V + 1)).astype(np.float32)
    for b in range(B):
        k = 5 * b
        for t in range(T):
            if (t + b) % blank_every == 0:
                rows[t, b, V] += margin
            else:
                rows[t, b, 1 + (k % plen)] += margin
                k += 1
    return rows


@pytest.mark.parametrize("chunk", [600, 16, 100])
def test_segment_starts_deep_inside_long_phrases(chunk):
    """Trajectories that stay deep inside a 40-token phrase: a segment start
    guessed from the root is wrong almost everywhere, so repairs run across
    many segments and workgroup boundaries."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    V, B, T = 64, 5, 600
    cm = np.concatenate([np.arange(V), [-1]]).astype(np.int32)
    phrase = list(range(1, 41))
    lists = [[phrase], [phrase, list(range(5, 30))], [list(range(1, 11))], [phrase]]
    rows = _phrase_following_rows(np.random.default_rng(7), T, B, V, 40)
    mids = np.array([0, 1, 2, 3, -1], np.int32)
    dec = BoostDecoder(lists, cm, token_w=1.0, end_bonus=2.0)
    say(f"[repair] long phrases, chunk={chunk}")
    gpu = gpu_greedy(dec, to_device_logits(rows), mids, chunk)
    graphs = {m: oracle.build_graph(l, cm, token_w=1.0, end_bonus=2.0) for m, l in enumerate(lists)}
    ref = oracle.greedy_decode(graphs, mids, rows[:, :, None, :], np.array([0, 0, 0, 0, -1], np.int32))
    compare_greedy(gpu, ref, range(B), ATOL)
    assert np.array_equal(gpu[3], ref[3])
    assert np.max(ref[1][:, 0]) >= 30          # the path really went deep


def test_segments_longer_than_the_kept_trajectory():
    """256 streams x 1100 steps in one call: one workgroup per stream with
    segments of 69 rows, and a 120-token phrase keeping repairs going past
    the first 64 rows of a segment."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    V, B, T, plen = 128, 256, 1100, 120
    cm = np.concatenate([np.arange(V), [-1]]).astype(np.int32)
    lists = [[list(range(1, plen + 1))], [list(range(1, 31)), list(range(40, 90))]]
    rows = _phrase_following_rows(np.random.default_rng(11), T, B, V, plen, blank_every=13)
    mids = (np.arange(B) % 2).astype(np.int32)
    dec = BoostDecoder(lists, cm, token_w=1.0, end_bonus=2.0)
    say("[repair] 256 x 1100, segments of 69 rows")
    gpu = gpu_greedy(dec, to_device_logits(rows), mids, T)
    sample = [0, 1, 2, 3, 100, 201, 254, 255]
    graphs = {m: oracle.build_graph(l, cm, token_w=1.0, end_bonus=2.0) for m, l in enumerate(lists)}
    sub = np.ascontiguousarray(rows[:, sample, None, :])
    ref = oracle.greedy_decode(graphs, mids[sample], sub, np.zeros(len(sample), np.int32))
    compare_greedy(gpu, ref, sample, ATOL, ref_streams=range(len(sample)))
    assert np.array_equal(gpu[3][sample], ref[3])
    assert np.max(ref[1][:, 0]) >= 100


def _shadow_case(extra):
    """A list where a suffix-chain child that a deeper child shadows has the
    larger psi: from state (1,1,2) the class-1 child (1,1,2,1) has psi 3 and
    the class-1 child (1,2,1) of its link (1,2) has psi 4 (commit reading:
    (1,1,2) is a phrase, so (1,1,2,1) holds 1 pending token; (1,2,1) holds 2).
    ``extra`` more children of (1,2) make the chain wider than one wave.
    Logits walk 1 1 2 1 9 blank, each stream out of phase."""
    V, B, T = 128, 3, 600
    cm = np.concatenate([np.arange(V), [-1]]).astype(np.int32)
    lst = [[1], [1, 1, 2], [1, 1, 2, 1, 9], [1, 2, 1, 9]] + [[1, 2, 20 + i] for i in range(extra)]
    rng = np.random.default_rng(3 + extra)
    rows = rng.normal(0.0, 0.1, size=(T, B, V + 1)).astype(np.float32)
    seq = [1, 1, 2, 1, 9, V]
    for b in range(B):
        for t in range(T):
            rows[t, b, seq[(t + b) % len(seq)]] += 3.0
    return V, B, T, cm, lst, rows


@pytest.mark.parametrize("extra", [0, 80])
@pytest.mark.parametrize("chunk", [16, 64, 600])
def test_shadowed_child_with_the_larger_psi(extra, chunk):
    """The best child over the whole suffix chain is a shadowed one: the step
    must take the deeper child of the same class (greedy, narrow and wide
    chains, short and long calls)."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    V, B, T, cm, lst, rows = _shadow_case(extra)
    g = oracle.build_graph(lst, cm, token_w=1.0, end_bonus=2.0)
    s112 = g.strings.index((1, 1, 2))
    deep, shallow = g.goto[s112][1], g.goto[g.link[s112]][1]
    assert g.psi64[shallow] > g.psi64[deep]
    mids = np.zeros(B, np.int32)
    dec = BoostDecoder([lst], cm, token_w=1.0, end_bonus=2.0)
    say(f"[shadow] extra={extra} chunk={chunk}")
    gpu = gpu_greedy(dec, to_device_logits(rows), mids, chunk)
    ref = oracle.greedy_decode({0: g}, mids, rows, np.zeros(B, np.int32))
    compare_greedy(gpu, ref, range(B), ATOL)
    assert np.sum(ref[1] == deep) >= 100  # the case really occurs


@pytest.mark.parametrize("extra", [0, 80])
def test_shadowed_child_with_the_larger_psi_beam(extra):
    """The same list and logits through the beam step (K = 3)."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    V, B, T, cm, lst, rows = _shadow_case(extra)
    K = 3
    rk = np.ascontiguousarray(np.repeat(rows[:, :, None, :], K, axis=2))
    g = oracle.build_graph(lst, cm, token_w=1.0, end_bonus=2.0)
    mids = np.zeros(B, np.int32)
    dec = BoostDecoder([lst], cm, token_w=1.0, end_bonus=2.0)
    say(f"[shadow] beam extra={extra}")
    gpu = gpu_beam(dec, to_device_logits(rk), mids, 16)
    st0, S0 = oracle.init_carry(mids, K)
    ref = oracle.beam_decode({0: g}, mids, rk, st0, S0)
    compare_beam(gpu, ref, range(B), ATOL)


def test_chunk_loop_graph_replay_matches_eager():
    """The streaming chunk loop captured in a HIP graph: every replay (with
    eager work and synchronisation in between) reproduces the eager outputs."""
    import torch
    from paper_2608_21343_amd import capi
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg = W.config_by_name("streaming")
    T, B, chunk = 96, cfg.B, 16
    dec = _decoder(cfg, W.phrases(cfg))
    logits = to_device_logits(W.logits(cfg, 0, T)[:, :, 0, :])
    mids, states, _ = dec.start(W.model_ids(cfg))
    tok = torch.empty((T, B), dtype=torch.int32, device="cuda")
    sst = torch.empty_like(tok)
    sc = torch.empty((T, B), dtype=torch.float32, device="cuda")

    def run():
        capi.tb_init_states(dec.arena, B, 1, mids, states)
        for ta in range(0, T, chunk):
            capi.tb_boost_step_greedy(dec.arena, logits[ta:ta + chunk], mids, states,
                                      tok[ta:ta + chunk], sst[ta:ta + chunk], sc[ta:ta + chunk])

    run()
    torch.cuda.synchronize()
    ref = [x.clone() for x in (tok, sst, sc, states)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    for rep in range(3):
        tok.fill_(-7)
        sst.fill_(-7)
        sc.fill_(0.5)
        states.fill_(3)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip((tok, sst, sc, states), ref):
            assert torch.equal(a, b), f"replay {rep} differs from the eager run"


BEAM_KERNEL = {"default": capi.BEAM_AUTO, "wide": capi.BEAM_NO_PIPE, "ref": capi.BEAM_REF}


@pytest.mark.parametrize("kernel", ["default", "ref"])
@pytest.mark.parametrize("K,dtype", [(1, "f32"), (2, "f32"), (3, "bf16"), (5, "bf16"), (8, "f32"),
                                     (20, "f32"), (32, "bf16")])
def test_beam_kernels_match_oracle_on_mixed_streams(kernel, K, dtype, restore_kernels):
    """Every beam kernel against the oracle: ragged V+1 = 301, model -1, an
    empty list and an out-of-range id (decoded unbiased, states -2)."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    capi.tb_debug_select_kernels(beam=BEAM_KERNEL[kernel])
    cfg, lists, rows = _small_case(6, B=6, V=300, K=K, T=40, dtype=dtype)
    lists = list(lists[:4]) + [[]]
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.array([0, -1, 4, 2, 99, 3], np.int32)
    say(f"[beam-{kernel}] K={K} {dtype}")
    gpu = gpu_beam(dec, to_device_logits(rows), mids, 40)
    ok = [0, 1, 2, 3, 5]
    graphs = oracle_graphs(cfg, lists, ok, mids)
    st0, S0 = oracle.init_carry(np.where(mids == 99, -1, mids), K)
    st0[mids == 99] = 0
    ref = oracle.beam_decode(graphs, np.where(mids == 99, -1, mids), rows, st0, S0)
    compare_beam(gpu, ref, ok, ATOL)
    # the out-of-range stream: unbiased beam search (tokens, parents and
    # accumulated scores of the oracle's model -1 run), states -2
    for i in (0, 1, 4):
        assert np.array_equal(gpu[i][:, 4], ref[i][:, 4]), i
    assert np.all(gpu[2][:, 4] == -2)


@pytest.mark.parametrize("kernel,V,K", [("default", 300, 3), ("default", 300, 8), ("ref", 300, 3),
                                        ("default", 2600, 4), ("wide", 2600, 4)])
def test_beam_bad_carried_states_decode_unbiased(kernel, V, K, restore_kernels):
    """A valid model id with a carried state out of range, TB_STATE_INVALID or
    TB_STATE_TIMEOUT in one of its slots: the stream is decoded without
    biasing (tokens, parents and scores of the oracle's model -1 run) and
    writes TB_STATE_INVALID, or TB_STATE_TIMEOUT when a slot carried it."""
    import torch
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    capi.tb_debug_select_kernels(beam=BEAM_KERNEL[kernel])
    cfg, lists, rows = _small_case(8, B=4, V=V, n_case=V // 10, K=K, T=20, dtype="f32")
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.array([0, 1, 2, 3], np.int32)
    say(f"[beam-bad-carry] {kernel} V+1={V + 1} K={K}")
    m, states, scores = dec.start(mids, K)
    carried = {1 * K + K - 1: 10 ** 6, 2 * K: capi.TB_STATE_TIMEOUT, 3 * K: capi.TB_STATE_INVALID}
    for i, v in carried.items():
        states[i] = v
    out = dec.beam(to_device_logits(rows), m, states, scores)
    torch.cuda.synchronize()
    gpu = [o.cpu().numpy() for o in out]
    graphs = oracle_graphs(cfg, lists, [0], mids)
    st0, S0 = oracle.init_carry(mids, K)
    ref = oracle.beam_decode(graphs, mids, rows, st0, S0, streams=[0])
    compare_beam(gpu, ref, [0], ATOL)
    free = np.array([0, -1, -1, -1], np.int32)
    st1, S1 = oracle.init_carry(free, K)
    ref1 = oracle.beam_decode(graphs, free, rows, st1, S1, streams=[1, 2, 3])
    for i in (0, 1, 4):
        assert np.array_equal(gpu[i][:, 1:], ref1[i][:, 1:]), i
    assert float(np.max(np.abs(gpu[3][:, 1:] - ref1[3][:, 1:]))) <= ATOL
    assert np.all(gpu[2][:, [1, 3]] == capi.TB_STATE_INVALID)
    assert np.all(gpu[2][:, 2] == capi.TB_STATE_TIMEOUT)


@pytest.mark.parametrize("kernel,V,K", [("default", 300, 3), ("ref", 300, 3), ("ref", 300, 12)])
def test_streaming_beam_bad_carried_states_decode_unbiased(kernel, V, K, restore_kernels):
    """The streaming beam with the carried states of the test above: the bad
    streams follow the oracle's streaming beam on model -1, chunk by chunk."""
    import torch
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    capi.tb_debug_select_kernels(beam=BEAM_KERNEL[kernel])
    cfg, lists, rows = _small_case(9, B=4, V=V, n_case=V // 10, K=K, T=24, dtype="f32")
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.array([0, 1, 2, 3], np.int32)
    say(f"[stream-beam-bad-carry] {kernel} V+1={V + 1} K={K}")
    carry = dec.start_beam_stream(mids, K, 64)
    carried = {1 * K + K - 1: 10 ** 6, 2 * K: capi.TB_STATE_TIMEOUT, 3 * K: capi.TB_STATE_INVALID}
    for i, v in carried.items():
        carry.states[i] = v
    graphs = oracle_graphs(cfg, lists, range(4), mids)
    ref = oracle.init_stream_carry(mids, K)
    free = np.array([0, -1, -1, -1], np.int32)
    ref1 = oracle.init_stream_carry(free, K)
    rows_dev = to_device_logits(rows)
    for t0 in range(0, cfg.T, 8):
        gpu = [o.cpu().numpy() for o in dec.beam_stream(rows_dev[t0:t0 + 8], carry)]
        want = oracle.beam_decode_stream(graphs, mids, rows[t0:t0 + 8], ref, tree_cap=64)
        compare_beam(gpu, want, [0], ATOL)
        want1 = oracle.beam_decode_stream(graphs, free, rows[t0:t0 + 8], ref1, tree_cap=64)
        for i in (0, 1, 4):
            assert np.array_equal(gpu[i][:, 1:], want1[i][:, 1:]), (t0, i)
        assert float(np.max(np.abs(gpu[3][:, 1:] - want1[3][:, 1:]))) <= ATOL
        assert np.all(gpu[2][:, [1, 3]] == capi.TB_STATE_INVALID)
        assert np.all(gpu[2][:, 2] == capi.TB_STATE_TIMEOUT)


GREEDY_KERNEL = {"default": capi.GREEDY_AUTO, "ref": capi.GREEDY_REF}


@pytest.mark.parametrize("kernel,V,chunk", [("default", 300, 16), ("default", 300, 200),
                                            ("default", 2600, 16), ("default", 2600, 200),
                                            ("ref", 300, 16)])
def test_greedy_bad_carried_states_decode_unbiased(kernel, V, chunk, restore_kernels):
    """Greedy with a valid model id and a carried state out of range,
    TB_STATE_INVALID or TB_STATE_TIMEOUT, through the short-call, segmented,
    wide-row and reference kernels: such a stream decodes without biasing and
    writes TB_STATE_INVALID (TB_STATE_TIMEOUT when it carried it)."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    capi.tb_debug_select_kernels(greedy=GREEDY_KERNEL[kernel])
    cfg, lists, rows = _small_case(10, B=4, V=V, n_case=V // 10, T=200)
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.array([0, 1, 2, 3], np.int32)
    say(f"[greedy-bad-carry] {kernel} V+1={V + 1} chunk={chunk}")
    s0 = np.array([0, 10 ** 6, capi.TB_STATE_TIMEOUT, capi.TB_STATE_INVALID], np.int32)
    tok, st, sc, carry = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, chunk,
                                    states0=s0)
    graphs = oracle_graphs(cfg, lists, [0], mids)
    ref = oracle.greedy_decode(graphs, mids, rows, np.zeros(4, np.int32), streams=[0])
    compare_greedy((tok, st, sc), ref, [0], ATOL)
    free = np.array([0, -1, -1, -1], np.int32)
    ref1 = oracle.greedy_decode(graphs, free, rows, np.full(4, -1, np.int32), streams=[1, 2, 3])
    assert np.array_equal(tok[:, 1:], ref1[0][:, 1:])
    assert float(np.max(np.abs(sc[:, 1:] - ref1[2][:, 1:]))) <= ATOL
    assert np.all(st[:, [1, 3]] == capi.TB_STATE_INVALID) and np.all(st[:, 2] == capi.TB_STATE_TIMEOUT)
    assert list(carry[1:]) == [capi.TB_STATE_INVALID, capi.TB_STATE_TIMEOUT, capi.TB_STATE_INVALID]


@pytest.mark.parametrize("kernel,V,K,chunk", [
    ("default", 300, 1, 16), ("default", 300, 1, 96), ("ref", 300, 1, 16),
    ("default", 2600, 1, 16), ("default", 2600, 1, 96),
    ("default", 300, 3, 96), ("default", 300, 8, 40), ("ref", 300, 3, 96),
    ("default", 2600, 4, 96), ("wide", 2600, 4, 96), ("stream", 300, 3, 32)])
def test_padded_row_stride_every_kernel(kernel, V, K, chunk, restore_kernels):
    """Rows farther apart than V+1 (seven values of 1e30 after each row, which
    any read of them would make win) through every greedy and beam kernel and
    the streaming beam, against the oracle on the unpadded rows."""
    import torch
    from paper_2608_21343_amd.decoder import BoostDecoder
    if K == 1:
        capi.tb_debug_select_kernels(greedy=GREEDY_KERNEL[kernel])
    elif kernel != "stream":
        capi.tb_debug_select_kernels(beam=BEAM_KERNEL[kernel])
    cfg, lists, rows = _small_case(11, B=4, V=V, n_case=V // 10, K=K, T=96)
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.array([0, 1, -1, 3], np.int32)
    T, B, V1 = cfg.T, cfg.B, cfg.Vp1
    say(f"[padded-stride] {kernel} V+1={V1} K={K} chunk={chunk}")
    pad = torch.full((T, B, K, V1 + 7), 1e30, dtype=torch.float32, device="cuda")
    pad[..., :V1] = torch.from_numpy(rows).cuda()
    view = pad[..., :V1]
    graphs = oracle_graphs(cfg, lists, range(B), mids)
    if K == 1:
        gpu = gpu_greedy(dec, view[:, :, 0, :], mids, chunk)
        ref = oracle.greedy_decode(graphs, mids, rows, np.where(mids >= 0, 0, -1).astype(np.int32))
        compare_greedy(gpu, ref, range(B), ATOL)
    elif kernel == "stream":
        carry = dec.start_beam_stream(mids, K, 128)
        want = oracle.init_stream_carry(mids, K)
        for t0 in range(0, T, chunk):
            got = [o.cpu().numpy() for o in dec.beam_stream(view[t0:t0 + chunk], carry)]
            exp = oracle.beam_decode_stream(graphs, mids, rows[t0:t0 + chunk], want, tree_cap=128)
            compare_beam(got, exp, range(B), ATOL)
    else:
        gpu = gpu_beam(dec, view, mids, chunk)
        st0, S0 = oracle.init_carry(mids, K)
        ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
        compare_beam(gpu, ref, range(B), ATOL)


@pytest.mark.parametrize("V", [2046, 2047, 2048])
@pytest.mark.parametrize("K,chunk", [(1, 16), (1, 100), (4, 100), (8, 50)])
def test_rows_at_the_wide_kernel_boundary(V, K, chunk):
    """V+1 = 2047, 2048 (the widest rows of the one-wave-per-row kernels) and
    2049 (the narrowest of the wide-row kernels), greedy in short and long
    calls and beam, against the oracle."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg, lists, rows = _small_case(12, B=4, V=V, n_case=V // 9, K=K, T=100, dtype="bf16")
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.array([0, 1, -1, 3], np.int32)
    say(f"[boundary] V+1={V + 1} K={K} chunk={chunk}")
    graphs = oracle_graphs(cfg, lists, range(cfg.B), mids)
    if K == 1:
        gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, chunk)
        ref = oracle.greedy_decode(graphs, mids, rows, np.where(mids >= 0, 0, -1).astype(np.int32))
        compare_greedy(gpu, ref, range(cfg.B), ATOL)
    else:
        gpu = gpu_beam(dec, to_device_logits(rows), mids, chunk)
        st0, S0 = oracle.init_carry(mids, K)
        ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
        compare_beam(gpu, ref, range(cfg.B), ATOL)


@pytest.mark.parametrize("V,K,dtype", [(1860, 8, "f32"), (1950, 4, "bf16"), (1983, 8, "bf16"),
                                       (1856, 2, "f32")])
def test_beam_rows_of_30_and_31_chunks(V, K, dtype):
    """Rows of 1857..1984 logits (30 or 31 chunks of 64 per lane, ragged last
    chunk) and the boundary below them, through the default beam kernel."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg, lists, rows = _small_case(7, B=6, V=V, n_case=V // 9, K=K, T=24, dtype=dtype)
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.array([0, 1, -1, 3, 4, 5], np.int32)
    say(f"[beam-chunks] V+1={V + 1} K={K} {dtype}")
    gpu = gpu_beam(dec, to_device_logits(rows), mids, 12)
    graphs = oracle_graphs(cfg, lists, range(cfg.B), mids)
    st0, S0 = oracle.init_carry(mids, K)
    ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
    compare_beam(gpu, ref, range(cfg.B), ATOL)


@pytest.mark.parametrize("kernel", ["default", "ref"])
def test_beam_inside_long_phrases(kernel, restore_kernels):
    """Beam hypotheses deep inside 40-token phrases (chains of several suffix
    states, override sets of dozens of classes)."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    capi.tb_debug_select_kernels(beam=BEAM_KERNEL[kernel])
    V, B, T, K = 64, 4, 200, 4
    cm = np.concatenate([np.arange(V), [-1]]).astype(np.int32)
    phrase = list(range(1, 41))
    lists = [[phrase, list(range(3, 20)), [5, 6, 7, 8]], [phrase, list(range(10, 50))],
             [list(range(1, 11)), [2, 3], [4, 5, 6]], [phrase]]
    base = _phrase_following_rows(np.random.default_rng(9), T, B, V, 40)
    rng = np.random.default_rng(10)
    rows = np.repeat(base[:, :, None, :], K, axis=2) + rng.normal(0, 0.3, (T, B, K, V + 1)).astype(np.float32)
    rows = np.ascontiguousarray(rows.astype(np.float32))
    mids = np.arange(B, dtype=np.int32)
    dec = BoostDecoder(lists, cm, token_w=1.0, end_bonus=2.0)
    say(f"[beam-{kernel}] long phrases")
    gpu = gpu_beam(dec, to_device_logits(rows), mids, 64)
    graphs = {m: oracle.build_graph(l, cm, token_w=1.0, end_bonus=2.0) for m, l in enumerate(lists)}
    st0, S0 = oracle.init_carry(mids, K)
    ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
    compare_beam(gpu, ref, range(B), ATOL)
    assert np.max(ref[2]) >= 20


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_wide_vocabulary_mixed_streams_and_chunks(dtype, restore_kernels):
    """Wide rows (V+1 = 3001, not a multiple of 256): the workgroup-segmented
    kernel against the oracle with model -1, an empty list and an
    out-of-range id, for whole calls (several segments per stream and the
    boundary fix-up) and chunked calls; tokens, states and carries equal the
    reference kernel's."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg = W.Config(107, "small", B=7, K=1, V=3000, T=96, chunk=96, dtype=dtype, n_phrases=200,
                   len_lo=1, len_hi=6, token_dist="zipf", zipf_s=1.1, logit_std=1.0,
                   blank_offset=1.0, n_case=300)
    lists = W.phrases(cfg)
    rows = W.logits(cfg)
    lists = list(lists[:5]) + [[]]
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.array([0, -1, 5, 3, 99, 4, 1], np.int32)
    dev = to_device_logits(rows[:, :, 0, :])
    ok = [0, 1, 2, 3, 5, 6]
    graphs = oracle_graphs(cfg, lists, ok, mids)
    st0 = np.array([0, -1, 0, 0, 0, 0, 0], np.int32)
    ref = oracle.greedy_decode(graphs, mids, rows, st0, streams=ok)
    outs = {}
    for chunk in (96, 37, 7, 1):
        say(f"[wide] {dtype} chunk={chunk}")
        gpu = gpu_greedy(dec, dev, mids, chunk)
        compare_greedy(gpu, ref, ok, ATOL)
        assert np.array_equal(gpu[3][ok], ref[3][ok])
        assert np.all(gpu[1][:, 1] == -1) and np.all(gpu[1][:, 4] == -2)
        assert np.all(gpu[1][:, 2] == 0)
        z = oracle.widen(rows[:, 4, 0, :])
        assert np.array_equal(gpu[0][:, 4], np.argmax(z, axis=1))
        outs[chunk] = gpu
    with capi.kernels(greedy=capi.GREEDY_REF):
        r = gpu_greedy(dec, dev, mids, 96)
    assert np.array_equal(outs[96][0], r[0]) and np.array_equal(outs[96][1], r[1])
    assert np.array_equal(outs[96][3], r[3])


def test_wide_vocabulary_segments_inside_long_phrases():
    """Wide rows whose boosted path stays inside a 40-token phrase: every
    guessed segment start is wrong, so the boundary fix-up recomputes across
    whole segments."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    V, B, T = 2600, 3, 400
    cm = np.concatenate([np.arange(V), [-1]]).astype(np.int32)
    phrase = list(range(1, 41))
    lists = [[phrase], [phrase, list(range(5, 30))], [list(range(1, 11))]]
    rows = _phrase_following_rows(np.random.default_rng(17), T, B, V, 40)
    mids = np.array([0, 1, 2], np.int32)
    dec = BoostDecoder(lists, cm, token_w=1.0, end_bonus=2.0)
    say("[wide] long phrases")
    gpu = gpu_greedy(dec, to_device_logits(rows), mids, T)
    graphs = {m: oracle.build_graph(l, cm, token_w=1.0, end_bonus=2.0) for m, l in enumerate(lists)}
    ref = oracle.greedy_decode(graphs, mids, rows[:, :, None, :], np.zeros(B, np.int32))
    compare_greedy(gpu, ref, range(B), ATOL)
    assert np.array_equal(gpu[3], ref[3])
    assert np.max(ref[1][:, 0]) >= 30


@pytest.mark.parametrize("kernel", ["default", "wide"])
@pytest.mark.parametrize("K,dtype", [(3, "f32"), (4, "bf16"), (8, "bf16")])
def test_wide_vocabulary_beam_mixed_streams(kernel, K, dtype, restore_kernels):
    """Beam kernels on wide rows (V+1 = 3001) against the oracle: model -1, an
    empty list and an out-of-range id (decoded unbiased, states -2), chunked
    calls equal one call, and the reference kernel agrees."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    capi.tb_debug_select_kernels(beam=BEAM_KERNEL[kernel])
    cfg = W.Config(108, "small", B=6, K=K, V=3000, T=40, chunk=40, dtype=dtype, n_phrases=200,
                   len_lo=1, len_hi=6, token_dist="zipf", zipf_s=1.1, logit_std=1.5,
                   blank_offset=0.0, n_case=300)
    lists = list(W.phrases(cfg)[:4]) + [[]]
    rows = W.logits(cfg)
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.array([0, -1, 4, 2, 99, 3], np.int32)
    dev = to_device_logits(rows)
    say(f"[wide-beam] K={K} {dtype}")
    gpu = gpu_beam(dec, dev, mids, 40)
    ok = [0, 1, 2, 3, 5]
    mm = np.where(mids == 99, -1, mids)
    graphs = oracle_graphs(cfg, lists, ok, mids)
    st0, S0 = oracle.init_carry(mm, K)
    st0[mids == 99] = 0
    ref = oracle.beam_decode(graphs, mm, rows, st0, S0)
    compare_beam(gpu, ref, ok, ATOL)
    for i in (0, 1, 4):
        assert np.array_equal(gpu[i][:, 4], ref[i][:, 4]), i
    assert np.all(gpu[2][:, 4] == -2)
    for ch in (7, 16):
        out = gpu_beam(dec, dev, mids, ch)
        for a, b in zip(gpu, out):
            assert np.array_equal(a, b), f"chunk {ch} differs"
    with capi.kernels(beam=capi.BEAM_REF):
        r = gpu_beam(dec, dev, mids, 40)
    for i in range(5):
        assert np.array_equal(gpu[i], r[i]) if i != 3 else np.max(np.abs(gpu[3] - r[3])) <= 1e-6


@pytest.mark.parametrize("kernel", ["default", "ref"])
@pytest.mark.parametrize("K", [1, 4, 7])
def test_beam_tiny_vocabulary(kernel, K, restore_kernels):
    """V+1 = 8 with K up to 7: fewer root moves than a row list holds, most
    candidates of a step in the K best, ties between equal logits."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    capi.tb_debug_select_kernels(beam=BEAM_KERNEL[kernel])
    V, B, T = 7, 3, 30
    cm = np.array([0, 0, 2, 3, 3, 5, 6, -1], np.int32)
    lists = [[[0, 2], [3, 5, 6], [2]], [[6, 6, 6]], []]
    rng = np.random.default_rng(21)
    rows = np.round(rng.normal(0, 1, (T, B, K, V + 1)) * 2) / 2  # many equal logits
    rows = np.ascontiguousarray(rows.astype(np.float32))
    mids = np.array([0, 1, 2], np.int32)
    dec = BoostDecoder(lists, cm, token_w=1.0, end_bonus=2.0)
    say(f"[beam-{kernel}] tiny vocabulary K={K}")
    gpu = gpu_beam(dec, to_device_logits(rows), mids, 11)
    graphs = {m: oracle.build_graph(l, cm, token_w=1.0, end_bonus=2.0) for m, l in enumerate(lists)}
    st0, S0 = oracle.init_carry(mids, K)
    ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
    compare_beam(gpu, ref, range(B), ATOL)


@pytest.mark.parametrize("kernel", ["default", "wide"])
@pytest.mark.parametrize("K,dtype", [(4, "bf16"), (2, "f32")])
def test_wide_vocabulary_beam_inside_long_phrases(kernel, K, dtype, restore_kernels):
    """Wide rows (V+1 = 2601) with hypotheses deep inside 40-token phrases
    whose tokens have the largest logits: most of a row's listed root moves
    are overridden, so the helper-wave kernel rescans rows too."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    capi.tb_debug_select_kernels(beam=BEAM_KERNEL[kernel])
    V, B, T = 2600, 4, 120
    cm = np.concatenate([np.arange(V), [-1]]).astype(np.int32)
    phrase = list(range(1, 41))
    lists = [[phrase, list(range(3, 20)), [5, 6, 7, 8]], [phrase, list(range(10, 50))],
             [list(range(1, 11)), [2, 3], [4, 5, 6]], [phrase]]
    base = _phrase_following_rows(np.random.default_rng(19), T, B, V, 40)
    rng = np.random.default_rng(20)
    rows = np.repeat(base[:, :, None, :], K, axis=2) + rng.normal(0, 0.3, (T, B, K, V + 1))
    rows = np.ascontiguousarray(rows.astype(np.float32))
    if dtype == "bf16":  # bfloat16 bits, rounded to nearest even
        from workloads.synth import _f32_to_bf16_bits
        rows = _f32_to_bf16_bits(rows)
    mids = np.arange(B, dtype=np.int32)
    dec = BoostDecoder(lists, cm, token_w=1.0, end_bonus=2.0)
    say(f"[beam-{kernel}] wide long phrases K={K} {dtype}")
    gpu = gpu_beam(dec, to_device_logits(rows), mids, 50)
    graphs = {m: oracle.build_graph(l, cm, token_w=1.0, end_bonus=2.0) for m, l in enumerate(lists)}
    st0, S0 = oracle.init_carry(mids, K)
    ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
    compare_beam(gpu, ref, range(B), ATOL)
    assert np.max(ref[2]) >= 20
