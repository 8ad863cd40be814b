"""tb_unregister_model_noalloc (the library's own scratch, no allocation)
against tb_unregister_model (a caller workspace), through the C ABI.

Two registries receive the same models; the same models are removed from
both, one with each entry point, two calls in a row (the second moves fewer
records). The device arenas must be byte-identical over the model table, the
used per-state ranges and the live per-model rows, and decoding through them
must give identical outputs. A removal whose records exceed the scratch is
rejected with TB_ENOMEM before any launch.
"""

import numpy as np
import pytest

import workloads as W
from paper_2608_21343_amd import capi
from tests.gpu_cases import gpu_greedy, say

pytestmark = pytest.mark.gpu


def _image(reg):
    import torch
    torch.cuda.synchronize()
    L = reg.arena.layout
    raw = reg.buf.cpu().numpy()
    pad = reg._base - reg.buf.data_ptr()
    return capi.image_arrays(raw[pad:pad + L.total_bytes], L)


def _same_arena(ra, rb, live):
    a, b = _image(ra), _image(rb)
    u = ra.used_states
    assert u == rb.used_states
    assert np.array_equal(a["model_off"], b["model_off"])
    assert np.array_equal(a["model_n"], b["model_n"])
    for k in ("first_child", "n_child", "link", "label", "phi", "psi"):
        assert np.array_equal(a[k][:u], b[k][:u]), k
    assert np.array_equal(a["arc_mem"][:2 * u], b["arc_mem"][:2 * u])
    assert np.array_equal(a["state_rec"][:u], b["state_rec"][:u])
    for k in ("root_psi", "root_dst", "value_tab"):
        assert np.array_equal(a[k][live], b[k][live]), k


def _decode(reg, rows_dev, mids):
    from paper_2608_21343_amd.decoder import BoostDecoder
    return gpu_greedy(BoostDecoder.for_arena(reg.arena), rows_dev, mids, 16)


def test_noalloc_removal_equals_workspace_removal():
    from paper_2608_21343_amd.decoder import to_device_logits
    cfg = W.config_by_name("streaming", B=12, T=48)
    cm = W.class_map(cfg)
    lists = W.phrases(cfg)
    g = capi.tb_compile_graphs(*W.phrase_csr(lists), 1.0, 2.0, cm)
    ra = capi.Registry(16, 2 * g.layout.n_states, cm)
    rb = capi.Registry(16, 2 * g.layout.n_states, cm)
    ids = ra.register(g)
    assert rb.register(g) == ids
    rows_dev = to_device_logits(W.logits(cfg)[:, :, 0, :])
    mids = np.arange(cfg.B, dtype=np.int32)
    live = list(ids)
    # first removal moves most of the arena, the second fewer records
    for victim in (ids[1], ids[9]):
        wa, wb = ra.workspace_bytes(victim), rb.workspace_bytes(victim)
        assert wa == wb
        say(f"[noalloc] removing id {victim}: {wa} bytes of records move")
        ra.unregister(victim)
        rb.unregister_noalloc(victim)
        live.remove(victim)
        _same_arena(ra, rb, live)
        oa, ob = _decode(ra, rows_dev, mids), _decode(rb, rows_dev, mids)
        for x, y in zip(oa, ob):
            assert np.array_equal(x, y)
    assert wa < ra.used_states * 44


def test_noalloc_rejects_records_beyond_its_scratch():
    cfg = W.Config(600, "big", B=1, K=1, V=1000, T=1, chunk=1, dtype="f32", n_phrases=120000,
                   len_lo=8, len_hi=8, token_dist="uniform", zipf_s=0.0, logit_std=1.0,
                   blank_offset=0.0, n_case=100)
    cm = W.class_map(cfg)
    big = W.phrases(cfg)[0]
    small = [np.array([1, 2, 3], np.int32)]
    gs = capi.tb_compile_graphs(*W.phrase_csr([small]), 1.0, 2.0, cm)
    gb = capi.tb_compile_graphs(*W.phrase_csr([big]), 1.0, 2.0, cm)
    assert gb.layout.n_states * 44 > (32 << 20)
    reg = capi.Registry(4, gs.layout.n_states + gb.layout.n_states, cm)
    sid = reg.register(gs)[0]
    bid = reg.register(gb)[0]
    before = (reg.used_states, reg.model(sid), reg.model(bid))
    with pytest.raises(capi.TbError) as e:
        reg.unregister_noalloc(sid)
    assert e.value.code == capi.TB_ENOMEM and "scratch" in str(e.value)
    assert (reg.used_states, reg.model(sid), reg.model(bid)) == before
    reg.unregister_noalloc(bid)          # the last model: nothing moves
    assert reg.model(bid)[1] == 0 and reg.used_states == gs.layout.n_states
