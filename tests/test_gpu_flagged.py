"""States whose packed 12-byte record cannot hold them (the record is flagged
and the kernels read the state from the arena's plain arrays instead):

* a state with 300 children (the record's child count has 8 bits);
* the states of a 300-token phrase whose potentials have more than 256
  distinct values (the record indexes a 256-entry value table);
* a model of more than 65,536 states (the record's first child and suffix
  link have 16 bits), so its deep states are flagged.

The logits walk each stream through the flagged states; greedy (short calls,
long calls, wide rows, reference kernel), beam (every kernel) and the
streaming beam against the oracle, and the compiled records are checked to be
flagged where expected. The long phrase's states also have value indexes
above 127 in their records (the top byte of a 32-bit word)."""

import numpy as np
import pytest

import oracle
from paper_2608_21343_amd import capi
from tests.gpu_cases import compare_beam, compare_greedy, gpu_beam, gpu_greedy, say

pytestmark = pytest.mark.gpu

ATOL = 1e-5
LONG = 300  # tokens of the long phrase (model 1)


def _lists(V, fan=300):
    rng = np.random.default_rng(11)
    # state (1, 2) with fan children: 300 is more than its record holds; 250
    # fills most of the beam kernel's override list (256) and, in the
    # short-call kernel's far-record instance, four children per lane; 30 is
    # an ordinary state
    fan = [[1, 2, 3 + i] for i in range(fan)]
    long = [[4 + (i % (V - 8)) for i in range(LONG)]]           # depths up to 300
    big = {tuple(int(t) for t in rng.integers(0, V, size=10)) for _ in range(7200)}
    big = [list(p) for p in sorted(big)]                        # about 70 k states
    small = [[5, 6, 7], [6, 7]]
    return [fan, long, big, small]


def _rows(V, T, K, lists, big_graph, seed):
    """Each stream follows its model's flagged states: the fan-out phrases, the
    long phrase from its start, and the big model's phrases that end in its
    last states (ids above 65,536), end to end."""
    rng = np.random.default_rng(seed)
    rows = rng.normal(0.0, 0.3, size=(T, 4, K, V + 1)).astype(np.float32)
    rows[..., V] += 0.5

    def plant(b, seq):
        for t, v in enumerate(seq[:T]):
            rows[t, b, :, int(v)] += 6.0

    plant(0, [v for i in range(T) for v in lists[0][(7 * i) % len(lists[0])]])
    plant(1, lists[1][0])
    deep = [big_graph.strings[x] for x in range(big_graph.n_states - 1, 65535, -37)]
    plant(2, [v for p in deep for v in p])
    plant(3, [5, 6, 7] * T)
    return np.ascontiguousarray(rows)


_CACHE = {}


def _setup(V, fan=300):
    from paper_2608_21343_amd.decoder import BoostDecoder
    if (V, fan) not in _CACHE:
        cm = np.concatenate([np.arange(V), [-1]]).astype(np.int32)
        lists = _lists(V, fan)
        dec = BoostDecoder(lists, cm, token_w=1.0, end_bonus=2.0)
        graphs = {m: oracle.build_graph(l, cm, token_w=1.0, end_bonus=2.0)
                  for m, l in enumerate(lists)}
        _CACHE[(V, fan)] = (cm, lists, dec, graphs)
    return _CACHE[(V, fan)]


def test_records_are_flagged_where_expected():
    _, lists, dec, graphs = _setup(1024)
    img = dec.graphs.host_image()
    a = capi.image_arrays(img, dec.graphs.layout)
    rec = a["state_rec"].reshape(-1, 3)
    flagged = (rec[:, 2] >> 31) != 0
    off, n = a["model_off"], a["model_n"]
    per_model = [int(flagged[off[m]:off[m] + n[m]].sum()) for m in range(4)]
    assert n[2] > 65536, n
    assert per_model[0] >= 1 and per_model[1] >= 1 and per_model[2] >= 1, per_model
    assert per_model[3] == 0, per_model


GREEDY_KERNEL = {"default": capi.GREEDY_AUTO, "ref": capi.GREEDY_REF}
BEAM_KERNEL = {"default": capi.BEAM_AUTO, "wide": capi.BEAM_NO_PIPE, "ref": capi.BEAM_REF}
T_STEPS = 320


@pytest.mark.parametrize("kernel,V,chunk,fan", [("default", 1024, 16, 300), ("default", 1024, 320, 300),
                                                ("default", 2600, 16, 300), ("default", 2600, 320, 300),
                                                ("ref", 1024, 16, 300), ("default", 1024, 16, 250),
                                                ("default", 1024, 320, 250)])
def test_greedy_through_flagged_records(kernel, V, chunk, fan, restore_kernels):
    from paper_2608_21343_amd.decoder import to_device_logits
    capi.tb_debug_select_kernels(greedy=GREEDY_KERNEL[kernel])
    cm, lists, dec, graphs = _setup(V, fan)
    rows = _rows(V, T_STEPS, 1, lists, graphs[2], 3)
    mids = np.arange(4, dtype=np.int32)
    say(f"[flagged] greedy {kernel} V+1={V + 1} chunk={chunk} fan-out={fan}")
    gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, chunk)
    ref = oracle.greedy_decode(graphs, mids, rows[:, :, 0, :], np.zeros(4, np.int32))
    compare_greedy(gpu, ref, range(4), ATOL)
    assert ref[1][:, 1].max() >= 290 and ref[1][:, 2].max() >= 65536


@pytest.mark.parametrize("kernel,V,K,fan", [("default", 1024, 4, 300), ("default", 1024, 8, 300),
                                            ("ref", 1024, 4, 300), ("default", 2600, 4, 300),
                                            ("wide", 2600, 4, 300), ("default", 1024, 4, 30),
                                            ("default", 1024, 8, 30), ("default", 2600, 4, 30),
                                            ("default", 1024, 4, 250), ("default", 1024, 8, 250)])
def test_beam_through_flagged_records(kernel, V, K, fan, restore_kernels):
    from paper_2608_21343_amd.decoder import to_device_logits
    capi.tb_debug_select_kernels(beam=BEAM_KERNEL[kernel])
    cm, lists, dec, graphs = _setup(V, fan)
    rows = _rows(V, T_STEPS, K, lists, graphs[2], 4)
    mids = np.arange(4, dtype=np.int32)
    say(f"[flagged] beam {kernel} V+1={V + 1} K={K} fan-out={fan}")
    gpu = gpu_beam(dec, to_device_logits(rows), mids, 80)
    st0, S0 = oracle.init_carry(mids, K)
    ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
    compare_beam(gpu, ref, range(4), ATOL)


@pytest.mark.parametrize("K", [4, 8])
def test_streaming_beam_through_flagged_records(K):
    """The streaming beam's merges take the psi of the merged state (a state
    of the long phrase, whose value index exceeds 127)."""
    from paper_2608_21343_amd.decoder import to_device_logits
    cm, lists, dec, graphs = _setup(1024, 30)
    rows = _rows(1024, T_STEPS, K, lists, graphs[2], 5)
    mids = np.arange(4, dtype=np.int32)
    say(f"[flagged] streaming beam K={K}")
    rows_dev = to_device_logits(rows)
    carry = dec.start_beam_stream(mids, K, 4096)
    want = oracle.init_stream_carry(mids, K)
    for t0 in range(0, T_STEPS, 80):
        got = [o.cpu().numpy() for o in dec.beam_stream(rows_dev[t0:t0 + 80], carry)]
        exp = oracle.beam_decode_stream(graphs, mids, rows[t0:t0 + 80], want, tree_cap=4096)
        compare_beam(got, exp, range(4), ATOL)


@pytest.mark.parametrize("chunk", [16, 320])
def test_greedy_wide_fan_out_in_small_models(chunk):
    """States with 100 and 200 children in models that fit the short-call
    kernel's LDS (its instance without far records: chains of 65 to 128
    children two per lane, larger ones level by level)."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    V = 1024
    cm = np.concatenate([np.arange(V), [-1]]).astype(np.int32)
    lists = [[[1, 2, 3 + i] for i in range(100)], [[1, 2, 3 + i] for i in range(200)],
             [[5, 6, 7], [6, 7]], [[1, 2, 3 + i] for i in range(70)] + [[2, 3 + i] for i in range(60)]]
    dec = BoostDecoder(lists, cm, token_w=1.0, end_bonus=2.0)
    graphs = {m: oracle.build_graph(l, cm, token_w=1.0, end_bonus=2.0) for m, l in enumerate(lists)}
    rng = np.random.default_rng(21)
    T = 320
    rows = rng.normal(0.0, 0.3, size=(T, 4, V + 1)).astype(np.float32)
    rows[..., V] += 0.5
    for b in range(4):
        seq = [v for i in range(T) for v in lists[b][(11 * i + b) % len(lists[b])]]
        for t, v in enumerate(seq[:T]):
            rows[t, b, int(v)] += 6.0
    mids = np.arange(4, dtype=np.int32)
    say(f"[flagged] greedy wide fan-out, small models, chunk={chunk}")
    gpu = gpu_greedy(dec, to_device_logits(rows), mids, chunk)
    ref = oracle.greedy_decode(graphs, mids, rows, np.zeros(4, np.int32))
    compare_greedy(gpu, ref, range(4), ATOL)


@pytest.mark.parametrize("K,chunk", [(1, 16), (1, 320), (4, 80), (8, 80)])
def test_suffix_chains_of_twenty_states(K, chunk):
    """A 24-token phrase listed with every one of its suffixes: deep in the
    phrase a state's suffix chain has up to 24 states with children, far
    beyond the chains the fast paths walk at once (the rest go level by
    level)."""
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    V = 300
    cm = np.concatenate([np.arange(V), [-1]]).astype(np.int32)
    ph = [10 + (7 * i) % 250 for i in range(24)]
    lists = [[ph[i:] for i in range(24)], [ph[i:] for i in range(0, 24, 3)] + [ph[:5]],
             [ph], [[5, 6, 7]]]
    dec = BoostDecoder(lists, cm, token_w=1.0, end_bonus=2.0)
    graphs = {m: oracle.build_graph(l, cm, token_w=1.0, end_bonus=2.0) for m, l in enumerate(lists)}
    rng = np.random.default_rng(31)
    T = 320
    rows = rng.normal(0.0, 0.3, size=(T, 4, K, V + 1)).astype(np.float32)
    rows[..., V] += 0.5
    for b in range(4):
        for t in range(T):
            rows[t, b, :, ph[(t + 3 * b) % 24]] += 6.0
    mids = np.arange(4, dtype=np.int32)
    say(f"[flagged] suffix chains K={K} chunk={chunk}")
    if K == 1:
        gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, chunk)
        ref = oracle.greedy_decode(graphs, mids, rows[:, :, 0, :], np.zeros(4, np.int32))
        compare_greedy(gpu, ref, range(4), ATOL)
        assert ref[1][:, 0].max() >= 20
    else:
        gpu = gpu_beam(dec, to_device_logits(rows), mids, chunk)
        st0, S0 = oracle.init_carry(mids, K)
        ref = oracle.beam_decode(graphs, mids, rows, st0, S0)
        compare_beam(gpu, ref, range(4), ATOL)
