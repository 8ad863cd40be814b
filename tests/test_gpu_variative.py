"""Decoding with variative BPE graphs on the GPU (Sec. II-A, Fig. 1c/1e,
Eq. (1)): lists written in characters, compiled by tb_compile_variative, and
decoded by the unchanged step kernels, against the oracle's variative graph
and its greedy, beam and streaming-beam steps.

The logits plant, every 16 steps, one phrase of the stream spelled by a random
segmentation into pieces in a random casing, so hypotheses run deep through
merged and character arcs. Tokens and states are compared bit for bit, step
scores within 1e-5, beam accumulated scores bit for bit.
"""

import numpy as np
import pytest

import oracle
import workloads.pieces as WP
from tests.gpu_cases import compare_beam, compare_greedy, gpu_beam, gpu_greedy, say

pytestmark = pytest.mark.gpu


def _case(B=8, K=1, V=400, T=96, dtype="f32", tau=1.0, n_phrases=40, seed=0):
    cfg = WP.piece_config("variative_small", index=30 + seed, B=B, K=K, V=V, T=T, dtype=dtype,
                          n_phrases=n_phrases, tau=tau)
    toks = WP.vocab(cfg)
    lists = WP.phrases(cfg)
    return cfg, toks, lists, WP.logits(cfg)


def _decoder(cfg, toks, lists, semantics=0):
    from paper_2608_21343_amd.decoder import BoostDecoder
    return BoostDecoder.variative(lists, toks, WP.LOWER, cfg.tau, token_w=cfg.token_w,
                                  end_bonus=cfg.end_bonus, semantics=semantics)


def _graphs(cfg, toks, lists, mids, semantics=0):
    return {int(m): oracle.build_variative_graph(toks, WP.LOWER, lists[int(m)],
                                                 token_w=cfg.token_w, end_bonus=cfg.end_bonus,
                                                 tau=cfg.tau, semantics=semantics)
            for m in set(mids.tolist()) if m >= 0}


@pytest.mark.parametrize("dtype,tau,semantics", [("f32", 1.0, 0), ("bf16", 0.0, 0),
                                                 ("f32", 2.0, 1)])
def test_greedy_on_variative_graphs(dtype, tau, semantics):
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg, toks, lists, rows = _case(dtype=dtype, tau=tau, seed=int(tau * 2) + semantics)
    mids = np.arange(cfg.B, dtype=np.int32)
    mids[3] = -1
    say(f"[variative-greedy] {dtype} tau={tau} semantics={semantics}")
    dec = _decoder(cfg, toks, lists, semantics)
    gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, 16)
    graphs = _graphs(cfg, toks, lists, mids, semantics)
    st0 = np.where(mids >= 0, 0, -1).astype(np.int32)
    ref = oracle.greedy_decode(graphs, mids, rows[:, :, 0, :], st0)
    compare_greedy(gpu, ref, range(cfg.B), 1e-5)
    # the planted spellings are matched: some streams reach deep states
    deep = max(len(graphs[m].strings[s]) for b, m in enumerate(mids) if m >= 0
               for s in ref[1][:, b])
    assert deep >= 6, deep


@pytest.mark.parametrize("K,dtype", [(4, "f32"), (8, "bf16")])
def test_beam_on_variative_graphs(K, dtype):
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg, toks, lists, rows = _case(K=K, dtype=dtype, T=64, seed=5 + K)
    mids = np.arange(cfg.B, dtype=np.int32)
    mids[1] = -1
    say(f"[variative-beam] K={K} {dtype}")
    dec = _decoder(cfg, toks, lists)
    gpu = gpu_beam(dec, to_device_logits(rows), mids, 16)
    graphs = _graphs(cfg, toks, lists, mids)
    st0, S0 = oracle.init_carry(mids, K)
    ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
    compare_beam(gpu, ref, range(cfg.B), 1e-5)


def test_streaming_beam_on_variative_graphs():
    import torch
    from paper_2608_21343_amd import capi
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg, toks, lists, rows = _case(K=4, T=48, seed=9)
    mids = np.arange(cfg.B, dtype=np.int32)
    dec = _decoder(cfg, toks, lists)
    graphs = _graphs(cfg, toks, lists, mids)
    rows_dev = to_device_logits(rows)
    carry = dec.start_beam_stream(mids, cfg.K, 1024)
    ref = oracle.init_stream_carry(mids, cfg.K)
    for t0 in range(0, cfg.T, 16):
        gpu = [o.cpu().numpy() for o in dec.beam_stream(rows_dev[t0:t0 + 16], carry)]
        want = oracle.beam_decode_stream(graphs, mids, rows[t0:t0 + 16], ref, tree_cap=1024)
        compare_beam(gpu, want, range(cfg.B), 1e-5)
    torch.cuda.synchronize()
    assert np.array_equal(carry.states.cpu().numpy().reshape(cfg.B, cfg.K), ref["states"])
    h = capi.hyp_fields(carry.hyps.cpu().numpy().reshape(cfg.B, cfg.K, 3))[0]
    for b in range(cfg.B):
        for j in range(cfg.K):
            assert int(h[b, j]) == capi.sequence_hash(ref["seqs"][b][j])


def test_variative_matches_class_graph_for_single_character_pieces():
    """A vocabulary of single characters only: the variative compile equals the
    class-graph compile of the same lists, and so do the decodes."""
    import torch
    from paper_2608_21343_amd import capi
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg, toks, lists, _ = _case(seed=11)
    chars = [(c,) for c in range(WP.N_CHARS)]
    cm = oracle.class_map_of(chars, WP.LOWER)
    lists = [[tuple(int(WP.LOWER[c]) for c in ph) for ph in lst] for lst in lists]
    a = BoostDecoder.variative(lists, chars, WP.LOWER, 1.0)
    b = BoostDecoder([[np.asarray(ph, np.int32) for ph in lst] for lst in lists], cm)
    ia, ib = a.graphs.host_image(), b.graphs.host_image()
    assert np.array_equal(ia, ib)
    rng = np.random.default_rng(3)
    rows = rng.standard_normal((32, cfg.B, WP.N_CHARS + 1)).astype(np.float32)
    mids = np.arange(cfg.B, dtype=np.int32)
    ga = gpu_greedy(a, to_device_logits(rows), mids, 16)
    gb = gpu_greedy(b, to_device_logits(rows), mids, 16)
    for x, y in zip(ga, gb):
        assert np.array_equal(x, y)


def test_variative_models_in_a_registry():
    """Variative graphs through the model lifecycle: register compiled lists,
    remove one (left-shift compaction; suffix links need not point to smaller
    ids here), then decode through the registry arena against the oracle."""
    from paper_2608_21343_amd import capi
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg, toks, lists, rows = _case(B=6, T=64, seed=13)
    cm = oracle.class_map_of(toks, WP.LOWER)
    reg = capi.Registry(max_models=6, max_states=200000, class_map=cm)

    def compiled(idx):
        sub = [lists[i] for i in idx]
        return BoostDecoder.variative(sub, toks, WP.LOWER, cfg.tau).graphs

    ids = reg.register(compiled([0, 1, 2])) + reg.register(compiled([3, 4, 5]))
    holds = dict(zip(ids, range(6)))
    victim = ids[1]
    reg.unregister(victim)
    del holds[victim]
    # stream j carries model id j (model ids[1] is free and decodes unbiased)
    mids = np.asarray(list(range(6)), np.int32)
    dec = BoostDecoder.for_arena(reg.arena)
    gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, 16)
    graphs = {m: oracle.build_variative_graph(toks, WP.LOWER, lists[holds[m]], tau=cfg.tau)
              for m in holds}
    ref_mids = np.asarray([m if m in holds else -1 for m in mids], np.int32)
    st0 = np.where(ref_mids >= 0, 0, -1).astype(np.int32)
    ref = oracle.greedy_decode(graphs, ref_mids, rows[:, :, 0, :], st0)
    assert np.array_equal(gpu[0], ref[0])
    live = [j for j in range(6) if mids[j] in holds]
    assert np.array_equal(gpu[1][:, live], ref[1][:, live])
    assert np.all(gpu[1][:, [j for j in range(6) if j not in live]] == capi.TB_STATE_INVALID)
    assert np.max(np.abs(gpu[2] - ref[2])) <= 1e-5
