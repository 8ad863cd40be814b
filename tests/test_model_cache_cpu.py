"""The host levels of the model cache (Sec. II-B, lifecycle paragraph):
compiled models in host memory (tb_graphs_cache_*) and on disk
(tb_graphs_save / tb_graphs_load). CPU only.

A cached compile must equal a fresh tb_compile_graphs byte for byte, whatever
mix of cached and new models a call holds; a file must load back to the same
image and layout, and every damaged file must be refused."""

import ctypes as C
import struct
import threading

import numpy as np
import pytest

import workloads as W
import workloads.pieces as WP
from paper_2608_21343_amd import capi

CFG = W.config_by_name("streaming", n_phrases=60)
CM = W.class_map(CFG)


def _lists(streams):
    return W.phrases(CFG, streams)


def _fresh(lists, w=None, bonus=None, scale=None, semantics=capi.TB_COMMIT):
    w = CFG.token_w if w is None else w
    bonus = CFG.end_bonus if bonus is None else bonus
    return capi.tb_compile_graphs(*W.phrase_csr(lists), w, bonus, CM, scale=scale,
                                  semantics=semantics)


def _cached(cache, lists, w=None, bonus=None, scale=None, semantics=capi.TB_COMMIT):
    w = CFG.token_w if w is None else w
    bonus = CFG.end_bonus if bonus is None else bonus
    return cache.compile(*W.phrase_csr(lists), w, bonus, scale=scale, semantics=semantics)


def _same(a: capi.Graphs, b: capi.Graphs):
    assert bytes(a.layout) == bytes(b.layout)
    assert np.array_equal(a.host_image(), b.host_image())


def test_cached_compile_equals_a_fresh_compile():
    lists = _lists(range(6))
    cache = capi.GraphsCache(CM)
    g1, h1 = _cached(cache, lists)
    assert h1 == 0
    _same(g1, _fresh(lists))
    g2, h2 = _cached(cache, lists)
    assert h2 == 6
    _same(g2, _fresh(lists))
    st = cache.stats()
    assert (st["hits"], st["misses"], st["models"], st["dropped"]) == (6, 6, 6, 0)
    assert st["bytes"] > 0
    # a mix of cached and new models, in another order, with a repeat
    mix = [lists[4], _lists([9])[0], lists[0], lists[4]]
    g3, h3 = _cached(cache, mix)
    assert h3 == 3
    _same(g3, _fresh(mix))


def test_every_compile_input_is_part_of_the_key():
    lists = _lists(range(3))
    cache = capi.GraphsCache(CM)
    _cached(cache, lists)
    base = _fresh(lists)
    for kw, want_hits in ((dict(w=np.asarray([CFG.token_w, 1.5, CFG.token_w], np.float32)), 2),
                          (dict(bonus=np.asarray([3.0, CFG.end_bonus, CFG.end_bonus], np.float32)), 2),
                          (dict(scale=np.asarray([1.0, 1.0, 0.5], np.float32)), 2),
                          (dict(semantics=capi.TB_PURE_POTENTIAL), 0)):
        g, h = _cached(cache, lists, **kw)
        assert h == want_hits, kw
        _same(g, _fresh(lists, **kw))
    # scale 1 is the default
    g, h = _cached(cache, lists, scale=np.ones(3, np.float32))
    assert h == 3
    _same(g, base)
    # one token of one phrase changed
    changed = [list(l) for l in lists]
    ph = np.array(changed[1][0], copy=True)
    ph[0] = (ph[0] + 1) % CFG.V
    changed[1][0] = ph
    g, h = _cached(cache, changed)
    assert h == 2
    _same(g, _fresh(changed))
    # an empty list and an empty phrase list are models too
    g, h = _cached(cache, [[], lists[0]])
    assert h == 1
    _same(g, _fresh([[], lists[0]]))


def test_least_recently_used_models_are_dropped():
    lists = _lists(range(5))
    probe = capi.GraphsCache(CM)
    _cached(probe, lists[:1])
    one = probe.stats()["bytes"]
    cache = capi.GraphsCache(CM, capacity_bytes=int(2.5 * one))
    _cached(cache, lists[:1])
    _cached(cache, lists[1:2])
    _cached(cache, lists[:1])  # model 0 is now the most recent
    _cached(cache, lists[2:3])  # drops model 1
    st = cache.stats()
    assert st["models"] == 2 and st["dropped"] >= 1 and st["bytes"] <= int(2.5 * one)
    _, h = _cached(cache, lists[:1])
    assert h == 1
    _, h = _cached(cache, lists[1:2])
    assert h == 0
    # a cache that holds nothing still compiles right
    none = capi.GraphsCache(CM, capacity_bytes=0)
    g, h = _cached(none, lists)
    g2, h2 = _cached(none, lists)
    assert h == h2 == 0 and none.stats()["models"] == 0
    _same(g2, _fresh(lists))


def test_concurrent_calls_on_one_cache():
    lists = _lists(range(8))
    want = _fresh(lists).host_image()
    cache = capi.GraphsCache(CM)
    errors, images = [], []

    def run(k):
        try:
            order = lists[k % 8:] + lists[:k % 8]
            g, _ = _cached(cache, order)
            images.append((k % 8, g.host_image()))
        except Exception as e:  # collected and re-raised below
            errors.append(e)

    threads = [threading.Thread(target=run, args=(k,)) for k in range(12)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for k, img in images:
        order = lists[k:] + lists[:k]
        assert np.array_equal(img, _fresh(order).host_image())
    g, h = _cached(cache, lists)
    assert h == 8
    assert np.array_equal(g.host_image(), want)


def test_cache_argument_errors():
    with pytest.raises(capi.TbError) as e:
        capi.GraphsCache(CM, capacity_bytes=-1)
    assert e.value.code == capi.TB_EINVAL
    bad = CM.copy()
    bad[-1] = 0
    with pytest.raises(capi.TbError) as e:
        capi.GraphsCache(bad)
    assert e.value.code == capi.TB_ERANGE
    cache = capi.GraphsCache(CM)
    lists = _lists(range(2))
    wrong = [list(l) for l in lists]
    wrong[1] = wrong[1] + [np.asarray([CFG.V], np.int32)]  # the blank inside a phrase
    with pytest.raises(capi.TbError) as e:
        _cached(cache, wrong)
    assert e.value.code == capi.TB_ERANGE
    # the failed call left the cache usable, and it kept the model that compiled
    g, h = _cached(cache, lists)
    assert h == 1
    _same(g, _fresh(lists))


# ---- files

HEAD = 32 + C.sizeof(capi.tb_arena_layout)  # tag, version, layout size, image size, checksum


def _fnv1a64(data: bytes) -> int:
    """64-bit FNV-1a from its definition (offset basis, then xor and multiply
    by the FNV prime per byte)."""
    h = 0xcbf29ce484222325
    for b in data:
        h = ((h ^ b) * 0x100000001b3) & 0xFFFFFFFFFFFFFFFF
    return h


def _variative():
    cfg = WP.piece_config("variative_small", B=3, n_phrases=12)
    toks = WP.vocab(cfg)
    mp, pp, pc = WP.phrase_csr(WP.phrases(cfg))
    tp, tc = WP.vocab_csr(toks)
    return capi.tb_compile_variative(mp, pp, pc, cfg.token_w, cfg.end_bonus, tp, tc, WP.LOWER,
                                     cfg.tau)


@pytest.mark.parametrize("kind", ["class", "variative"])
def test_save_and_load(tmp_path, kind):
    g = _fresh(_lists(range(4))) if kind == "class" else _variative()
    path = tmp_path / "m.tbg"
    capi.tb_graphs_save(g, path)
    assert path.stat().st_size == HEAD + g.layout.total_bytes
    assert not list(tmp_path.glob("*.tmp*"))
    back = capi.tb_graphs_load(path)
    _same(g, back)
    capi.tb_validate_image(back.host_image(), back.layout)
    # the stored checksum is FNV-1a of the image
    raw = path.read_bytes()
    assert struct.unpack_from("<Q", raw, 24)[0] == _fnv1a64(raw[HEAD:])
    # saving over an existing file replaces it
    g2 = _fresh(_lists([7]))
    capi.tb_graphs_save(g2, path)
    _same(g2, capi.tb_graphs_load(path))


def _refused(path, code):
    with pytest.raises(capi.TbError) as e:
        capi.tb_graphs_load(path)
    assert e.value.code == code, e.value


def test_damaged_files_are_refused(tmp_path):
    g = _fresh(_lists(range(2)))
    good = tmp_path / "good.tbg"
    capi.tb_graphs_save(g, good)
    raw = bytearray(good.read_bytes())
    lay = capi.tb_arena_layout.from_buffer_copy(bytes(raw[32:HEAD]))

    def write(name, data):
        p = tmp_path / name
        p.write_bytes(bytes(data))
        return p

    def with_checksum(data):
        data = bytearray(data)
        struct.pack_into("<Q", data, 24, _fnv1a64(bytes(data[HEAD:])))
        return data

    _refused(tmp_path / "missing.tbg", capi.TB_EIO)
    _refused(write("empty.tbg", b""), capi.TB_ERANGE)
    bad = bytearray(raw)
    bad[0:8] = b"NOTGRAPH"
    _refused(write("tag.tbg", bad), capi.TB_ERANGE)
    bad = bytearray(raw)
    struct.pack_into("<I", bad, 8, 2)  # another version
    _refused(write("version.tbg", bad), capi.TB_ERANGE)
    _refused(write("short.tbg", raw[:-5]), capi.TB_ERANGE)
    _refused(write("long.tbg", raw + b"\0"), capi.TB_ERANGE)
    # a flipped byte in the image: the checksum catches it
    bad = bytearray(raw)
    bad[HEAD + lay.off_link + 4 * 3] ^= 0x01
    _refused(write("flip.tbg", bad), capi.TB_ERANGE)
    # the same flip with a matching checksum: the image validation catches it
    # (a suffix link out of its model or into a cycle, or a record mismatch)
    bad = bytearray(raw)
    struct.pack_into("<i", bad, HEAD + lay.off_link + 4 * 3, 10 ** 6)
    _refused(write("link.tbg", with_checksum(bad)), capi.TB_ERANGE)
    # a layout maximum that disagrees with the image
    for field in ("max_override", "max_children"):
        l2 = capi.tb_arena_layout.from_buffer_copy(bytes(raw[32:HEAD]))
        setattr(l2, field, getattr(l2, field) - 1)
        bad = bytearray(raw)
        bad[32:HEAD] = bytes(l2)
        _refused(write(f"{field}.tbg", bad), capi.TB_ERANGE)
    # an offset that is not the one the counts imply
    l2 = capi.tb_arena_layout.from_buffer_copy(bytes(raw[32:HEAD]))
    l2.off_psi += 256
    bad = bytearray(raw)
    bad[32:HEAD] = bytes(l2)
    _refused(write("offset.tbg", bad), capi.TB_ERANGE)
    # counts that no image has
    l2 = capi.tb_arena_layout.from_buffer_copy(bytes(raw[32:HEAD]))
    l2.n_models = 0
    bad = bytearray(raw)
    bad[32:HEAD] = bytes(l2)
    _refused(write("count.tbg", bad), capi.TB_ERANGE)
    # the good file still loads
    _same(g, capi.tb_graphs_load(good))


def test_save_errors(tmp_path):
    g = _fresh(_lists(range(1)))
    with pytest.raises(capi.TbError) as e:
        capi.tb_graphs_save(g, tmp_path / "no_such_dir" / "m.tbg")
    assert e.value.code == capi.TB_EIO
