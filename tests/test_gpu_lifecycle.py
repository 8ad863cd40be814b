"""Model lifecycle on the GPU (Sec. II-B): models added to a registry arena by
appending, removed by a left-shift compaction of the later state ranges, with
stable ids.

After every register / unregister of a sequence:
* each live model's records in the device arena equal a fresh
  tb_compile_graphs of its list (every per-state array over its range, its
  root row and value table under its id);
* greedy decoding through the registry arena equals the oracle built from the
  live lists (a free id and model -1 decode without biasing);
* across a removal, streams on the other models decode bit-identically.
"""

import numpy as np
import pytest

import oracle
import workloads as W
from paper_2608_21343_amd import capi
from tests.gpu_cases import gpu_beam, gpu_greedy, say

pytestmark = pytest.mark.gpu


def _setup(n_lists=8, V=300, n_case=40, seed=0):
    cfg = W.Config(500 + seed, "life", B=n_lists, K=1, V=V, T=48, chunk=16, dtype="f32",
                   n_phrases=80, len_lo=1, len_hi=7, token_dist="zipf", zipf_s=1.1,
                   logit_std=1.0, blank_offset=1.0, n_case=n_case)
    lists = W.phrases(cfg)
    lists[3] = []                      # an empty list (root-only model)
    return cfg, lists, W.class_map(cfg)


def _compile(lists, cm):
    return capi.tb_compile_graphs(*W.phrase_csr(lists), 1.0, 2.0, cm)


class Model:
    """Host view of the registry: which list each live id holds."""

    def __init__(self, reg, cm):
        self.reg, self.cm, self.live = reg, cm, {}

    def register(self, lists, idx):
        ids = self.reg.register(_compile([lists[i] for i in idx], self.cm))
        for i, j in zip(idx, ids):
            assert j not in self.live
            self.live[j] = i
        return ids

    def unregister(self, model_id):
        self.reg.unregister(model_id)
        del self.live[model_id]


def _check_records(model, lists):
    import torch
    reg = model.reg
    torch.cuda.synchronize()
    L = reg.arena.layout
    raw = reg.buf.cpu().numpy()
    pad = reg._base - reg.buf.data_ptr()
    a = capi.image_arrays(raw[pad:pad + L.total_bytes], L)
    used = 0
    for mid, li in model.live.items():
        f, n = reg.model(mid)
        g = _compile([lists[li]], model.cm)
        b = capi.image_arrays(g.host_image(), g.layout)
        assert n == b["model_n"][0] and n > 0
        for k in ("first_child", "n_child", "link", "label", "phi", "psi"):
            assert np.array_equal(a[k][f:f + n], b[k][:n]), (mid, k)
        assert np.array_equal(a["arc_mem"][2 * f:2 * (f + n)], b["arc_mem"][:2 * n]), mid
        assert np.array_equal(a["state_rec"][f:f + n], b["state_rec"][:n]), mid
        for k in ("root_psi", "root_dst", "value_tab"):
            assert np.array_equal(a[k][mid], b[k][0]), (mid, k)
        assert a["model_off"][mid] == f and a["model_n"][mid] == n
        used += n
    for mid in range(reg.max_models):
        if mid not in model.live:
            assert a["model_n"][mid] == 0 and reg.model(mid)[1] == 0
    assert used == reg.used_states
    # the live ranges tile [0, used) without gaps, in some order
    spans = sorted(reg.model(m) for m in model.live)
    pos = 0
    for f, n in spans:
        assert f == pos
        pos += n


def _decode(model, lists, rows_dev, rows):
    """Stream j carries model id j (live or free), the last stream model -1;
    checked against the oracle (a free id decodes without biasing)."""
    from paper_2608_21343_amd.decoder import BoostDecoder
    M = model.reg.max_models
    mids = np.array(list(range(M)) + [-1], np.int32)
    B = len(mids)
    dec = BoostDecoder.for_arena(model.reg.arena)
    gpu = gpu_greedy(dec, rows_dev[:, :B].contiguous(), mids, 16)
    graphs = {m: oracle.build_graph(lists[model.live[m]], model.cm, token_w=1.0, end_bonus=2.0)
              for m in model.live}
    ref_mids = np.array([m if m in model.live else -1 for m in mids], np.int32)
    st0 = np.where(ref_mids >= 0, 0, -1).astype(np.int32)
    ref = oracle.greedy_decode(graphs, ref_mids, rows[:, :B], st0)
    assert np.array_equal(gpu[0], ref[0]), "tokens differ from the oracle"
    live = [j for j in range(B) if mids[j] in model.live or mids[j] == -1]
    free = [j for j in range(B) if j not in live]
    assert np.array_equal(gpu[1][:, live], ref[1][:, live]), "states differ"
    assert np.all(gpu[1][:, free] == capi.TB_STATE_INVALID)
    assert np.max(np.abs(gpu[2] - ref[2])) <= 1e-5
    return gpu


def test_register_unregister_sequence():
    import torch
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg, lists, cm = _setup()
    reg = capi.Registry(max_models=6, max_states=20000, class_map=cm)
    model = Model(reg, cm)
    rows = W.logits(cfg, 0, 48, streams=range(cfg.B))[:, :, 0, :]
    rows = np.ascontiguousarray(np.concatenate([rows, rows[:, :2]], axis=1))  # up to 10 streams
    rows_dev = to_device_logits(rows)
    steps = [("reg", [0, 1, 2]), ("reg", [3]), ("unreg", 1), ("reg", [4]), ("unreg", 0),
             ("reg", [5, 6]), ("unreg", 6), ("unreg", 3), ("reg", [7, 1]), ("unreg", 2)]
    for op, arg in steps:
        if op == "reg":
            ids = model.register(lists, arg)
            say(f"[lifecycle] registered lists {arg} as ids {ids}")
        else:
            victim = [m for m, li in model.live.items() if li == arg][0]
            keep = sorted(m for m in model.live if m != victim)
            out_b = _decode(model, lists, rows_dev, rows)
            model.unregister(victim)
            say(f"[lifecycle] removed list {arg} (id {victim}); used states {reg.used_states}")
            out_a = _decode(model, lists, rows_dev, rows)
            # streams on the other models are bit-identical across the removal
            for x, y in zip(out_b[:3], out_a[:3]):
                assert np.array_equal(x[:, keep], y[:, keep])
        _check_records(model, lists)
        _decode(model, lists, rows_dev, rows)


def test_unregister_rejects_a_small_workspace_and_changes_nothing():
    import torch
    cfg, lists, cm = _setup(seed=1)
    reg = capi.Registry(max_models=4, max_states=10000, class_map=cm)
    model = Model(reg, cm)
    ids = model.register(lists, [0, 1, 2])
    need = reg.workspace_bytes(ids[0])
    assert need == 44 * (reg.used_states - reg.model(ids[0])[1])
    small = torch.empty(need - 4, dtype=torch.uint8, device="cuda")
    with pytest.raises(capi.TbError) as e:
        reg.unregister(ids[0], workspace=small)
    assert e.value.code == capi.TB_ENOMEM
    _check_records(model, lists)
    assert reg.workspace_bytes(ids[2]) == 0          # the last model: nothing moves
    model.unregister(ids[2])
    _check_records(model, lists)
    with pytest.raises(capi.TbError) as e:
        reg.unregister(ids[2])
    assert e.value.code == capi.TB_EINVAL


def test_capacity_and_class_map_checks():
    cfg, lists, cm = _setup(seed=2)
    reg = capi.Registry(max_models=2, max_states=600, class_map=cm)
    model = Model(reg, cm)
    with pytest.raises(capi.TbError) as e:        # three models, two ids
        model.register(lists, [0, 1, 2])
    assert e.value.code == capi.TB_ENOMEM and reg.used_states == 0
    g = _compile([lists[0]], cm)
    if g.layout.n_states <= 600:
        model.register(lists, [0])
    big = _compile([lists[1], lists[2], lists[4]], cm)
    with pytest.raises(capi.TbError):
        reg.register(big)
    other = cm.copy()
    other[[0, 1]] = other[[1, 0]]
    with pytest.raises(capi.TbError) as e:
        reg.register(capi.tb_compile_graphs(*W.phrase_csr([lists[5]]), 1.0, 2.0, other))
    assert e.value.code == capi.TB_EINVAL
    _check_records(model, lists)


def test_beam_through_the_registry_after_compaction():
    from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits
    cfg, lists, cm = _setup(seed=3)
    reg = capi.Registry(max_models=5, max_states=20000, class_map=cm)
    model = Model(reg, cm)
    model.register(lists, [0, 1, 2, 4])
    victim = [m for m, li in model.live.items() if li == 1][0]
    model.unregister(victim)
    K = 3
    mids = np.array(sorted(model.live), np.int32)
    rows = W.logits(cfg, 0, 40, streams=range(len(mids)))
    rk = np.ascontiguousarray(np.repeat(rows, K, axis=2))
    dec = BoostDecoder.for_arena(reg.arena)
    gpu = gpu_beam(dec, to_device_logits(rk), mids, 16)
    graphs = {m: oracle.build_graph(lists[model.live[m]], cm, token_w=1.0, end_bonus=2.0)
              for m in model.live}
    st0, S0 = oracle.init_carry(mids, K)
    ref = oracle.beam_decode(graphs, mids, rk, st0, S0)
    from tests.gpu_cases import compare_beam
    compare_beam(gpu, ref, range(len(mids)), 1e-5)


def test_models_from_the_host_cache_and_from_files(tmp_path):
    """The paper's cache levels feeding the registry: models taken from the
    host-memory cache and loaded from files give the same arena records and
    decodes as freshly compiled ones."""
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg, lists, cm = _setup(seed=4)
    reg = capi.Registry(max_models=6, max_states=20000, class_map=cm)
    model = Model(reg, cm)
    cache = capi.GraphsCache(cm)
    rows = W.logits(cfg, 0, 48, streams=range(cfg.B))[:, :, 0, :]
    rows_dev = to_device_logits(rows)

    def add(graphs, idx):
        ids = reg.register(graphs)
        for i, j in zip(idx, ids):
            model.live[j] = i
        return ids

    g, hits = cache.compile(*W.phrase_csr([lists[0], lists[1]]), 1.0, 2.0)
    assert hits == 0
    add(g, [0, 1])
    path = tmp_path / "list2.tbg"
    capi.tb_graphs_save(_compile([lists[2]], cm), path)
    add(capi.tb_graphs_load(path), [2])
    say("[lifecycle] lists 0, 1 from the cache, 2 from a file")
    _check_records(model, lists)
    _decode(model, lists, rows_dev, rows)
    victim = [m for m, li in model.live.items() if li == 0][0]
    model.unregister(victim)
    g, hits = cache.compile(*W.phrase_csr([lists[0], lists[4]]), 1.0, 2.0)
    assert hits == 1
    add(g, [0, 4])
    say("[lifecycle] list 0 again from the cache after its removal")
    _check_records(model, lists)
    _decode(model, lists, rows_dev, rows)
