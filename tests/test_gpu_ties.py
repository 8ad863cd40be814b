"""GPU parity on greedy rows with tied keys (ties go to the lowest token id).

Logits are multiples of 0.5 and every potential is an integer (w = 1, end
bonus 2), so boosted keys tie often. The oracle's key vectors are inspected on
the CPU to make sure the ties that matter really occur at the selected
maximum:

* two case variants of one class (same boost, equal logits);
* the blank against a token (the blank, id V, must lose);
* an override child of the suffix chain against a root move.

Each case runs through the short-call kernel (chunks of 16), one long call
(segments over several workgroups and the boundary fix-up), the wide-row
kernels (V+1 > 2048) and the reference kernel.
"""

import numpy as np
import pytest

import oracle
import workloads as W
from oracle.decode import _keys
from paper_2608_21343_amd import capi
from tests.gpu_cases import compare_greedy, gpu_greedy, oracle_graphs, say

pytestmark = pytest.mark.gpu
ATOL = 1e-5


def _tie_case(V, n_case, B=6, T=640, seed=0):
    cfg = W.Config(300 + seed, "ties", B=B, K=1, V=V, T=T, chunk=T, dtype="f32", n_phrases=60,
                   len_lo=1, len_hi=5, token_dist="zipf", zipf_s=1.3, logit_std=1.0,
                   blank_offset=0.0, n_case=n_case)
    lists = W.phrases(cfg)
    rng = np.random.default_rng(1000 + seed)
    rows = (rng.integers(-4, 3, size=(T, B, V + 1)) * 0.5).astype(np.float32)
    rows[:, :, : 3 * n_case] += np.float32(1.5)     # cased (phrase-heavy) tokens compete
    rows[:, :, V] = (rng.integers(2, 10, size=(T, B)) * 0.5).astype(np.float32)
    # copy the logit of a class's lowercase member onto its upper-case variant
    # in some rows, so that case variants tie exactly
    cv = rng.random((T, B)) < 0.5
    c = rng.integers(0, n_case, size=(T, B))
    t_i, b_i = np.nonzero(cv)
    rows[t_i, b_i, c[t_i, b_i] + n_case] = rows[t_i, b_i, c[t_i, b_i]]
    return cfg, lists, rows


def _tie_census(cfg, graphs, mids, rows, ref):
    """Counts of rows whose maximum key is shared by (case variants, blank and
    a token, an override child and a root move), replaying the oracle's path."""
    cm = W.class_map(cfg)
    V = cfg.V
    n = {"case": 0, "blank": 0, "override_vs_root": 0}
    for b in range(cfg.B):
        g = graphs.get(int(mids[b]))
        s = 0
        for t in range(cfg.T):
            z = rows[t, b]
            key, dst, _ = _keys(g, s, z)
            top = np.nonzero(key == key.max())[0]
            if len(top) > 1:
                toks = [v for v in top if v < V]
                if V in top and toks:
                    n["blank"] += 1
                cls = [int(cm[v]) for v in toks]
                if len(set(cls)) < len(cls):
                    n["case"] += 1
                if g is not None and toks:
                    root = g.token_row(0)
                    over = [v for v in toks if dst[v] != root[v]]
                    plain = [v for v in toks if dst[v] == root[v]]
                    if over and plain:
                        n["override_vs_root"] += 1
            s = int(ref[1][t, b])
    return n


CASES = {"narrow": (300, 40), "wide": (2600, 300)}


@pytest.mark.parametrize("width", ["narrow", "wide"])
def test_greedy_ties_go_to_the_lowest_index(width):
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    V, n_case = CASES[width]
    cfg, lists, rows = _tie_case(V, n_case, seed=0 if width == "narrow" else 1)
    mids = W.model_ids(cfg)
    graphs = oracle_graphs(cfg, lists, range(cfg.B), mids)
    ref = oracle.greedy_decode(graphs, mids, rows, np.zeros(cfg.B, np.int32))
    census = _tie_census(cfg, graphs, mids, rows, ref)
    say(f"[ties] {width}: ties at the maximum {census}")
    assert census["case"] >= 20 and census["blank"] >= 20 and census["override_vs_root"] >= 5
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    dev = to_device_logits(rows)
    for chunk in (16, cfg.T):           # short calls, then one call (segments + fix-up)
        say(f"[ties] {width}: chunk {chunk}")
        gpu = gpu_greedy(dec, dev, mids, chunk)
        compare_greedy(gpu, ref, range(cfg.B), ATOL)
        assert np.array_equal(gpu[3], ref[3])
    with capi.kernels(greedy=capi.GREEDY_REF):
        say(f"[ties] {width}: reference kernel")
        gpu = gpu_greedy(dec, dev, mids, 64)
        compare_greedy(gpu, ref, range(cfg.B), ATOL)


@pytest.mark.parametrize("K", [2, 4])
def test_beam_ties_go_to_the_lowest_flat_index(K):
    """The same tied rows through the beam step (every slot reads the stream's
    row): equal candidates are ordered by flat index k*(V+1)+v."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    from tests.gpu_cases import compare_beam, gpu_beam
    cfg, lists, rows = _tie_case(300, 40, B=4, T=96, seed=2)
    rk = np.ascontiguousarray(np.repeat(rows[:, :, None, :], K, axis=2))
    mids = W.model_ids(cfg)
    graphs = oracle_graphs(cfg, lists, range(cfg.B), mids)
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    say(f"[ties] beam K={K}")
    gpu = gpu_beam(dec, to_device_logits(rk), mids, 16)
    st0, S0 = oracle.init_carry(mids, K)
    ref = oracle.beam_decode(graphs, mids, rk, st0, S0)
    compare_beam(gpu, ref, range(cfg.B), ATOL)
