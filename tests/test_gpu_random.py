"""Seeded random configurations through the automatic kernel choice, against
the oracle: vocabulary sizes on both sides of every dispatch boundary (one
token, one wave, 2048 logits, wide rows), beams of 1 to 12 hypotheses, any
chunk length, fp32 and bf16, case classes of three or five members, empty
and nested lists, unbiased streams, rows
farther apart than V+1, and phrases planted in the logits so that states go
deep. Greedy, plain beam and
streaming beam, every stream compared element by element."""

import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_cases import compare_beam, compare_greedy, gpu_beam, gpu_greedy, say
from workloads.synth import _f32_to_bf16_bits

pytestmark = pytest.mark.gpu

ATOL = 1e-5
N_CASES = 120


def _case(seed):
    rng = np.random.default_rng(7000 + seed)
    V = int(rng.choice([1, 2, 5, 63, 64, 65, 200, 1023, 1024, 2047, 2048, 2600, 4200]))
    K = int(rng.choice([1, 1, 2, 3, 4, 5, 8, 12]))
    K = min(K, V + 1)
    T = int(rng.integers(1, 49))
    cfg = W.Config(7000 + seed, "random", B=int(rng.integers(1, 7)), K=K, V=V, T=T,
                   chunk=int(rng.integers(1, T + 1)), dtype=str(rng.choice(["f32", "bf16"])),
                   n_phrases=int(rng.integers(1, 60)), len_lo=1, len_hi=int(rng.integers(1, 9)),
                   token_dist=str(rng.choice(["uniform", "zipf"])), zipf_s=1.1,
                   logit_std=float(rng.choice([0.5, 1.0, 2.0])),
                   blank_offset=float(rng.choice([0.0, 1.0])), n_case=int(rng.integers(0, V // 3 + 1)))
    lists = [list(lst) for lst in W.phrases(cfg)]
    lists[0].append(lists[0][0][:1])  # a nested (or repeated) phrase
    for b in range(1, cfg.B):
        if rng.random() < 0.15:
            lists[b] = []  # an empty list: root only, no biasing
    mids = np.arange(cfg.B, dtype=np.int32)
    mids[rng.random(cfg.B) < 0.2] = -1
    rows = W.logits(cfg.__class__(**{**cfg.__dict__, "dtype": "f32"}))
    for b in range(cfg.B):
        if mids[b] < 0 or not len(lists[b]):
            continue
        t = int(rng.integers(0, 3))
        while True:
            ph = lists[b][int(rng.integers(len(lists[b])))]
            if t + len(ph) > T:
                break
            for i, v in enumerate(ph):
                rows[t + i, b, :, int(v)] += np.float32(4.0)
            t += len(ph) + int(rng.integers(0, 4))
    if cfg.dtype == "bf16":
        rows = _f32_to_bf16_bits(rows)
    pad = int(rng.choice([0, 0, 1, 5, 64]))  # row stride V+1+pad
    cm = W.class_map(cfg)
    if V >= 10 and rng.random() < 0.3:
        # classes of five members (more than an arc record holds inline)
        n5 = int(rng.integers(1, V // 5 + 1))
        cm = np.arange(V + 1, dtype=np.int32)
        for k in range(1, 5):
            cm[k * n5:(k + 1) * n5] = np.arange(n5)
        cm[V] = -1
    return (cfg, lists, mids, np.ascontiguousarray(rows), str(rng.choice(["plain", "stream"])),
            pad, cm)


def _device_rows(rows, pad):
    """rows on the device, each row followed by pad values of 1e30 that no
    kernel may read."""
    import torch
    from paper_2608_21343_amd.decoder import to_device_logits
    dev = to_device_logits(rows)
    if pad == 0:
        return dev
    full = torch.empty(dev.shape[:-1] + (dev.shape[-1] + pad,), dtype=dev.dtype, device=dev.device)
    full.fill_(1e30)
    full[..., :dev.shape[-1]] = dev
    return full[..., :dev.shape[-1]]


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_configuration(seed):
    from paper_2608_21343_amd.decoder import BoostDecoder
    cfg, lists, mids, rows, beam_kind, pad, cm = _case(seed)
    dec = BoostDecoder(lists, cm, token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    graphs = {int(m): oracle.build_graph(lists[m], cm, token_w=cfg.token_w,
                                         end_bonus=cfg.end_bonus)
              for m in set(mids.tolist()) if m >= 0}
    kind = "greedy" if cfg.K == 1 else beam_kind
    say(f"[random {seed}] {kind} V+1={cfg.Vp1} K={cfg.K} B={cfg.B} T={cfg.T} chunk={cfg.chunk} "
        f"{cfg.dtype} phrases={cfg.n_phrases} pad={pad}")
    if cfg.K == 1:
        gpu = gpu_greedy(dec, _device_rows(rows, pad)[:, :, 0, :], mids, cfg.chunk)
        st0 = np.where(mids >= 0, 0, -1).astype(np.int32)
        ref = oracle.greedy_decode(graphs, mids, rows[:, :, 0, :], st0)
        compare_greedy(gpu, ref, range(cfg.B), ATOL)
    elif kind == "plain":
        gpu = gpu_beam(dec, _device_rows(rows, pad), mids, cfg.chunk)
        st0, S0 = oracle.init_carry(mids, cfg.K)
        ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
        compare_beam(gpu, ref, range(cfg.B), ATOL)
    else:
        rows_dev = _device_rows(rows, pad)
        carry = dec.start_beam_stream(mids, cfg.K, 64)
        want = oracle.init_stream_carry(mids, cfg.K)
        for t0 in range(0, cfg.T, cfg.chunk):
            got = [o.cpu().numpy() for o in dec.beam_stream(rows_dev[t0:t0 + cfg.chunk], carry)]
            exp = oracle.beam_decode_stream(graphs, mids, rows[t0:t0 + cfg.chunk], want,
                                            tree_cap=64)
            compare_beam(got, exp, range(cfg.B), ATOL)


def _variative_case(seed):
    import workloads.pieces as WP
    rng = np.random.default_rng(9000 + seed)
    K = int(rng.choice([1, 1, 2, 4, 8]))
    T = int(rng.integers(1, 41))
    cfg = WP.piece_config("variative_small", index=9000 + seed, B=int(rng.integers(1, 6)), K=K,
                          V=int(rng.choice([WP.N_CHARS, 120, 400, 1100, 2100])), T=T,
                          chunk=int(rng.integers(1, T + 1)), dtype=str(rng.choice(["f32", "bf16"])),
                          n_phrases=int(rng.integers(1, 25)), n_lexicon=600,
                          tau=float(rng.choice([0.0, 1.0, 2.0])))
    return cfg, int(rng.integers(0, 2)), str(rng.choice(["plain", "stream"]))


@pytest.mark.parametrize("seed", range(N_CASES // 4))
def test_random_variative_configuration(seed):
    """Variative BPE graphs (lists in characters over a piece vocabulary,
    Eq. (1) potentials, both readings of the potentials) in random
    configurations, against the oracle's variative graph."""
    import workloads.pieces as WP
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg, semantics, beam_kind = _variative_case(seed)
    toks, lists, rows = WP.vocab(cfg), WP.phrases(cfg), WP.logits(cfg)
    mids = np.arange(cfg.B, dtype=np.int32)
    if cfg.B > 1:
        mids[-1] = -1
    kind = "greedy" if cfg.K == 1 else beam_kind
    say(f"[random variative {seed}] {kind} pieces={cfg.V} K={cfg.K} B={cfg.B} T={cfg.T} "
        f"chunk={cfg.chunk} {cfg.dtype} tau={cfg.tau} semantics={semantics}")
    dec = BoostDecoder.variative(lists, toks, WP.LOWER, cfg.tau, token_w=cfg.token_w,
                                 end_bonus=cfg.end_bonus, semantics=semantics)
    graphs = {int(m): oracle.build_variative_graph(toks, WP.LOWER, lists[int(m)],
                                                   token_w=cfg.token_w, end_bonus=cfg.end_bonus,
                                                   tau=cfg.tau, semantics=semantics)
              for m in set(mids.tolist()) if m >= 0}
    if cfg.K == 1:
        gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, cfg.chunk)
        st0 = np.where(mids >= 0, 0, -1).astype(np.int32)
        ref = oracle.greedy_decode(graphs, mids, rows[:, :, 0, :], st0)
        compare_greedy(gpu, ref, range(cfg.B), ATOL)
    elif kind == "plain":
        gpu = gpu_beam(dec, to_device_logits(rows), mids, cfg.chunk)
        st0, S0 = oracle.init_carry(mids, cfg.K)
        ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
        compare_beam(gpu, ref, range(cfg.B), ATOL)
    else:
        rows_dev = to_device_logits(rows)
        carry = dec.start_beam_stream(mids, cfg.K, 64)
        want = oracle.init_stream_carry(mids, cfg.K)
        for t0 in range(0, cfg.T, cfg.chunk):
            got = [o.cpu().numpy() for o in dec.beam_stream(rows_dev[t0:t0 + cfg.chunk], carry)]
            exp = oracle.beam_decode_stream(graphs, mids, rows[t0:t0 + cfg.chunk], want,
                                            tree_cap=64)
            compare_beam(got, exp, range(cfg.B), ATOL)


@pytest.mark.parametrize("K,chunk", [(1, 16), (1, 40), (3, 40)])
def test_many_streams(K, chunk):
    """700 streams (more workgroups than CUs; one segment per stream in long
    greedy calls), 70 models shared by the streams, against the oracle."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg = W.Config(7500 + K, "many", B=70, K=K, V=64, T=40, chunk=chunk, dtype="f32",
                   n_phrases=30, len_lo=1, len_hi=5, token_dist="zipf", zipf_s=1.1,
                   logit_std=1.0, blank_offset=0.5, n_case=10)
    lists = W.phrases(cfg)
    cm = W.class_map(cfg)
    B = 700
    rng = np.random.default_rng(7600 + K)
    mids = rng.integers(-1, 70, size=B).astype(np.int32)
    rows = rng.normal(0.0, 1.0, size=(40, B, K, 65)).astype(np.float32)
    for b in range(B):
        if mids[b] >= 0:
            ph = lists[mids[b]][int(rng.integers(len(lists[mids[b]])))]
            t0 = int(rng.integers(0, 30))
            for i, v in enumerate(ph):
                if t0 + i < 40:
                    rows[t0 + i, b, :, int(v)] += 4.0
    dec = BoostDecoder(lists, cm, token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    graphs = {int(m): oracle.build_graph(lists[m], cm, token_w=cfg.token_w,
                                         end_bonus=cfg.end_bonus)
              for m in set(mids.tolist()) if m >= 0}
    say(f"[many streams] B={B} K={K} chunk={chunk}")
    if K == 1:
        gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, chunk)
        ref = oracle.greedy_decode(graphs, mids, rows[:, :, 0, :],
                                   np.where(mids >= 0, 0, -1).astype(np.int32))
        compare_greedy(gpu, ref, range(B), ATOL)
    else:
        gpu = gpu_beam(dec, to_device_logits(rows), mids, chunk)
        st0, S0 = oracle.init_carry(mids, K)
        ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
        compare_beam(gpu, ref, range(B), ATOL)


@pytest.mark.parametrize("V,K,dtype", [(300, 1, "f32"), (300, 1, "bf16"), (300, 4, "f32"),
                                       (300, 8, "bf16"), (2600, 1, "f32"), (2600, 4, "bf16")])
def test_masked_logits(V, K, dtype):
    """Rows with -inf logits (masked tokens): about a third of every row, and
    rows where only the blank and one or two tokens are finite."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg = W.Config(7700 + V + K, "masked", B=5, K=K, V=V, T=48, chunk=16, dtype="f32",
                   n_phrases=40, len_lo=1, len_hi=5, token_dist="zipf", zipf_s=1.1,
                   logit_std=1.0, blank_offset=0.5, n_case=V // 10)
    lists = W.phrases(cfg)
    cm = W.class_map(cfg)
    rng = np.random.default_rng(7800 + V + K)
    rows = W.logits(cfg)
    mask = rng.random(rows.shape) < 0.33
    mask[..., V] = False
    sparse = rng.random(rows.shape[:3]) < 0.15
    keep = rng.integers(0, V, size=rows.shape[:3] + (2,))
    for idx in zip(*np.nonzero(sparse)):
        mask[idx] = True
        mask[idx][keep[idx]] = False
        mask[idx][V] = False
    rows[mask] = -np.inf
    for b in range(5):  # planted phrases stay finite
        ph = lists[b][0]
        for i, v in enumerate(ph):
            rows[10 + i, b, :, int(v)] = 6.0
    if dtype == "bf16":
        rows = _f32_to_bf16_bits(rows)
    rows = np.ascontiguousarray(rows)
    mids = np.array([0, 1, 2, -1, 4], np.int32)
    dec = BoostDecoder(lists, cm, token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    graphs = {m: oracle.build_graph(lists[m], cm, token_w=cfg.token_w, end_bonus=cfg.end_bonus)
              for m in (0, 1, 2, 4)}
    say(f"[masked] V+1={V + 1} K={K} {dtype}")
    if K == 1:
        gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, 16)
        ref = oracle.greedy_decode(graphs, mids, rows[:, :, 0, :],
                                   np.where(mids >= 0, 0, -1).astype(np.int32))
        compare_greedy(gpu, ref, range(5), ATOL)
    else:
        gpu = gpu_beam(dec, to_device_logits(rows), mids, 16)
        st0, S0 = oracle.init_carry(mids, K)
        ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
        compare_beam(gpu, ref, range(5), ATOL)
