"""Streaming beam with hypothesis recombination on the GPU (Sec. II-C:
hypotheses carried across chunks in a flattened tree, continued, merged and
pruned), against the oracle's streaming beam.

Every case compares, per step, tokens, parents, states and accumulated scores
bit for bit and step scores within 1e-5; after every chunk, the carried states
and scores bit for bit, every slot's tb_hyp record against the oracle's label
sequence (hash, prefix hash, last label, node) and every stream's tree.

Workloads are the beam workload's shape family with a blank offset that makes
blank and label extensions of one parent survive together, so merges happen
on most steps; recombine=False is checked against the plain beam entry point.
The chunk loop is also captured in a HIP graph and replayed.
"""

import numpy as np
import pytest

import oracle
import workloads as W
from paper_2608_21343_amd import capi
from tests.gpu_cases import say

pytestmark = pytest.mark.gpu


def _cfg(seed, B, K, V, T, dtype="f32", blank_offset=3.0, logit_std=1.0, n_phrases=120):
    return W.Config(700 + seed, "stream_beam", B=B, K=K, V=V, T=T, chunk=16, dtype=dtype,
                    n_phrases=n_phrases, len_lo=1, len_hi=6, token_dist="zipf", zipf_s=1.1,
                    logit_std=logit_std, blank_offset=blank_offset, n_case=max(1, V // 9))


def _graphs(cfg, mids):
    lists, cm = W.phrases(cfg), W.class_map(cfg)
    return {m: oracle.build_graph(lists[m], cm, token_w=cfg.token_w, end_bonus=cfg.end_bonus)
            for m in set(int(x) for x in mids) if m >= 0}


def _setup(cfg, mids):
    from paper_2608_21343_amd.decoder import BoostDecoder
    dec = BoostDecoder(W.phrases(cfg), W.class_map(cfg), token_w=cfg.token_w,
                       end_bonus=cfg.end_bonus)
    return dec, _graphs(cfg, mids)


def _check_carry(carry_dev, ref, B, K, cap):
    import torch
    torch.cuda.synchronize()
    assert np.array_equal(carry_dev.states.cpu().numpy().reshape(B, K), ref["states"])
    assert np.array_equal(carry_dev.scores.cpu().numpy().reshape(B, K), ref["scores"])
    h, hp, last, node = capi.hyp_fields(carry_dev.hyps.cpu().numpy().reshape(B, K, 3))
    assert np.array_equal(node, ref["nodes"]), "tree nodes differ"
    for b in range(B):
        for j in range(K):
            seq = ref["seqs"][b][j]
            assert int(h[b, j]) == capi.sequence_hash(seq), (b, j)
            assert int(hp[b, j]) == (capi.sequence_hash(seq[:-1]) if seq else 0), (b, j)
            assert int(last[b, j]) == (seq[-1] if seq else -1), (b, j)
    tl = carry_dev.tree_len.cpu().numpy()
    tree = carry_dev.tree.cpu().numpy() if carry_dev.tree is not None else None
    for b in range(B):
        want = ref["trees"][b]
        assert tl[b] == len(want) <= cap, (b, tl[b], len(want))
        if want:
            assert np.array_equal(tree[b, :tl[b]], np.asarray(want, np.int32)), b


def _run(cfg, mids, chunk, recombine=True, cap=4096, check_every_chunk=True):
    import torch
    from paper_2608_21343_amd.decoder import to_device_logits
    B, K, T = cfg.B, cfg.K, cfg.T
    dec, graphs = _setup(cfg, mids)
    rows = W.logits(cfg)
    rows_dev = to_device_logits(rows)
    carry = dec.start_beam_stream(mids, K, cap)
    ref = oracle.init_stream_carry(mids, K)
    for t0 in range(0, T, chunk):
        t1 = min(T, t0 + chunk)
        gpu = [o.cpu().numpy() for o in dec.beam_stream(rows_dev[t0:t1], carry, recombine)]
        want = oracle.beam_decode_stream(graphs, mids, rows[t0:t1], ref, recombine=recombine,
                                         tree_cap=cap)
        for i, n in enumerate(["tok", "parent", "state"]):
            bad = np.nonzero(gpu[i] != want[i])
            assert bad[0].size == 0, f"{n} mismatch at (t, b, k) {list(zip(*bad))[:5]} (t0={t0})"
        assert np.array_equal(gpu[4], want[4]), f"accumulated score not bit-exact (t0={t0})"
        err = float(np.max(np.abs(gpu[3] - want[3])))
        assert err <= 1e-5, f"step score error {err}"
        if check_every_chunk or t1 == T:
            _check_carry(carry, ref, B, K, cap)
    return rows, rows_dev, ref


def _merges(cfg, mids):
    """Steps at which recombination changes the oracle's result (so that the
    merge path is exercised)."""
    graphs = _graphs(cfg, mids)
    rows = W.logits(cfg, 0, 24)
    a = oracle.beam_decode_stream(graphs, mids, rows, oracle.init_stream_carry(mids, cfg.K))
    b = oracle.beam_decode_stream(graphs, mids, rows, oracle.init_stream_carry(mids, cfg.K),
                                  recombine=False)
    return int(np.sum(np.any(a[4] != b[4], axis=2)))


@pytest.mark.parametrize("K,V,dtype", [(8, 1024, "f32"), (4, 300, "bf16"), (2, 1000, "f32"),
                                       (8, 1999, "bf16"), (8, 1600, "f32"), (6, 1900, "f32"),
                                       (1, 63, "f32"),
                                       (5, 64, "f32")])
def test_stream_beam_matches_the_oracle(K, V, dtype):
    cfg = _cfg(K + V, B=12, K=K, V=V, T=48, dtype=dtype)
    mids = np.arange(cfg.B, dtype=np.int32)
    mids[5] = -1                      # an unbiased stream
    say(f"[stream-beam] K={K} V={V} {dtype}: merges on {_merges(cfg, mids)} stream-steps")
    _run(cfg, mids, chunk=16)


@pytest.mark.parametrize("K,V,dtype", [(4, 3000, "f32"), (12, 500, "f32"), (3, 5000, "bf16"),
                                       (32, 300, "f32")])
def test_stream_beam_on_the_reference_kernel(K, V, dtype):
    """Rows wider than 2048 and beams wider than 8: the reference kernel's
    streaming stage."""
    cfg = _cfg(K * 7 + V, B=6, K=K, V=V, T=32, dtype=dtype)
    mids = np.arange(cfg.B, dtype=np.int32)
    mids[2] = -1
    say(f"[stream-beam-ref] K={K} V={V} {dtype}: merges on {_merges(cfg, mids)} stream-steps")
    _run(cfg, mids, chunk=16)


def test_stream_beam_reference_kernel_forced(restore_kernels):
    """The reference kernel's streaming stage on a row the fast kernel would
    take, forced through the test hook."""
    from paper_2608_21343_amd import capi
    capi.tb_debug_select_kernels(beam=capi.BEAM_REF)
    cfg = _cfg(77, B=8, K=8, V=700, T=32)
    mids = np.arange(cfg.B, dtype=np.int32)
    _run(cfg, mids, chunk=16)


def test_recombination_is_exercised():
    cfg = _cfg(1, B=12, K=8, V=1024, T=24)
    assert _merges(cfg, np.arange(cfg.B, dtype=np.int32)) >= 20


def test_without_recombination_equals_the_plain_beam():
    import torch
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg = _cfg(2, B=10, K=8, V=700, T=40)
    mids = np.arange(cfg.B, dtype=np.int32)
    dec, _ = _setup(cfg, mids)
    rows_dev = to_device_logits(W.logits(cfg))
    carry = dec.start_beam_stream(mids, cfg.K, 512)
    m2, st, sc = dec.start(mids, cfg.K)
    for t0 in range(0, cfg.T, 16):
        a = dec.beam_stream(rows_dev[t0:t0 + 16], carry, recombine=False)
        b = dec.beam(rows_dev[t0:t0 + 16], m2, st, sc)
        torch.cuda.synchronize()
        for x, y in zip(a, b):
            assert torch.equal(x, y)
    assert torch.equal(carry.states, st) and torch.equal(carry.scores, sc)


def test_tree_capacity_marks_records_that_do_not_fit():
    cfg = _cfg(3, B=6, K=4, V=200, T=40, blank_offset=1.0)
    mids = np.arange(cfg.B, dtype=np.int32)
    rows, _, ref = _run(cfg, mids, chunk=13, cap=25)
    assert any(len(t) == 25 for t in ref["trees"]) and np.any(ref["nodes"] == -2)


def test_no_tree_storage():
    cfg = _cfg(4, B=4, K=4, V=128, T=20)
    mids = np.arange(cfg.B, dtype=np.int32)
    _run(cfg, mids, chunk=20, cap=0)


def test_chunking_does_not_change_results():
    import torch
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg = _cfg(5, B=8, K=8, V=512, T=45)
    mids = np.arange(cfg.B, dtype=np.int32)
    dec, _ = _setup(cfg, mids)
    rows_dev = to_device_logits(W.logits(cfg))
    outs = []
    for chunk in (45, 7, 1):
        c = dec.start_beam_stream(mids, cfg.K, 1024)
        parts = [dec.beam_stream(rows_dev[t0:t0 + chunk], c) for t0 in range(0, cfg.T, chunk)]
        torch.cuda.synchronize()
        outs.append(([torch.cat([p[i] for p in parts]) for i in range(5)], c))
    (o0, c0) = outs[0]
    for o, c in outs[1:]:
        for x, y in zip(o0, o):
            assert torch.equal(x, y)
        for x, y in ((c0.states, c.states), (c0.scores, c.scores), (c0.hyps, c.hyps),
                     (c0.tree_len, c.tree_len), (c0.tree, c.tree)):
            assert torch.equal(x, y)


def test_argument_errors():
    import torch
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg = _cfg(6, B=2, K=4, V=100, T=4)
    mids = np.arange(cfg.B, dtype=np.int32)
    dec, _ = _setup(cfg, mids)
    rows_dev = to_device_logits(W.logits(cfg))
    c = dec.start_beam_stream(mids, 4, 16)

    def outs(K):
        return [torch.empty((4, 2, K), dtype=torch.int32, device="cuda") for _ in range(3)] + \
               [torch.empty((4, 2, K), dtype=torch.float32, device="cuda") for _ in range(2)]

    with pytest.raises(ValueError):   # a short hypothesis buffer
        capi.tb_boost_step_beam_stream(dec.arena, rows_dev, c.mids, c.states, c.scores,
                                       c.hyps[:3], c.tree, c.tree_len, *outs(4))
    # K beyond TB_MAX_BEAM
    Kx = capi.TB_MAX_BEAM + 1
    cfgx = _cfg(6, B=2, K=Kx, V=100, T=4)
    rowsx = to_device_logits(W.logits(cfgx))
    cx = dec.start_beam_stream(mids, 4, 16)
    with pytest.raises(capi.TbError) as e:
        capi.tb_boost_step_beam_stream(dec.arena, rowsx, cx.mids,
                                       torch.zeros(2 * Kx, dtype=torch.int32, device="cuda"),
                                       torch.zeros(2 * Kx, dtype=torch.float32, device="cuda"),
                                       torch.zeros((2 * Kx, 3), dtype=torch.int64, device="cuda"),
                                       cx.tree, cx.tree_len, *outs(Kx))
    assert e.value.code == capi.TB_EINVAL


def _graph_replay(stream_beam: bool):
    import torch
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg = _cfg(7, B=16, K=8, V=1024, T=64)
    chunk = 16
    mids = np.arange(cfg.B, dtype=np.int32)
    dec, _ = _setup(cfg, mids)
    rows_dev = to_device_logits(W.logits(cfg))
    i32 = dict(dtype=torch.int32, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    shape = (chunk, cfg.B, cfg.K)

    def outs():
        return tuple([torch.empty(shape, **i32) for _ in range(3)] +
                     [torch.empty(shape, **f32) for _ in range(2)])

    def step(inp, carry, out):
        if stream_beam:
            dec.beam_stream(inp, carry, out=out)
        else:
            dec.beam(inp, carry[0], carry[1], carry[2], out=out)

    def start():
        return dec.start_beam_stream(mids, cfg.K, 512) if stream_beam else dec.start(mids, cfg.K)

    # eager reference
    ce, eager = start(), []
    for t0 in range(0, cfg.T, chunk):
        o = outs()
        step(rows_dev[t0:t0 + chunk], ce, o)
        eager.append([x.clone() for x in o])
    torch.cuda.synchronize()
    # captured: one graph over a static input, replayed per chunk
    cg = start()
    static_in = torch.empty_like(rows_dev[:chunk])
    static_out = outs()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(static_in, cg, static_out)
    for i, t0 in enumerate(range(0, cfg.T, chunk)):
        static_in.copy_(rows_dev[t0:t0 + chunk])
        g.replay()
        torch.cuda.synchronize()
        for x, y in zip(static_out, eager[i]):
            assert torch.equal(x, y), f"replay {i} differs from the eager call"
    if stream_beam:
        for x, y in ((ce.states, cg.states), (ce.scores, cg.scores), (ce.hyps, cg.hyps),
                     (ce.tree, cg.tree), (ce.tree_len, cg.tree_len)):
            assert torch.equal(x, y)
    else:
        assert torch.equal(ce[1], cg[1]) and torch.equal(ce[2], cg[2])


def test_stream_beam_chunk_loop_in_a_hip_graph():
    _graph_replay(True)


def test_plain_beam_chunk_loop_in_a_hip_graph():
    _graph_replay(False)
