"""The host compiler of the variative BPE graph (tb_compile_variative) against
the oracle's variative graph, array by array, on the synthetic piece
vocabulary; image validation; argument errors. CPU only."""

import numpy as np
import pytest

import oracle
import workloads.pieces as WP
from oracle.graph import COMMIT, PURE_POTENTIAL
from paper_2608_21343_amd import capi


def _compile(cfg, lists, toks, tau, scale=None, semantics=COMMIT):
    mp, pp, pc = WP.phrase_csr(lists)
    tp, tc = WP.vocab_csr(toks)
    return capi.tb_compile_variative(mp, pp, pc, cfg.token_w, cfg.end_bonus, tp, tc, WP.LOWER,
                                     tau, scale=scale, semantics=semantics)


def _expected(g, V):
    n = g.n_states
    fc = np.zeros(n, np.int32)
    nc = np.zeros(n, np.int32)
    lab = np.full(n, -1, np.int32)
    for s in range(n):
        kids = g.goto[s]
        nc[s] = len(kids)
        fc[s] = min(kids.values()) if kids else 0
        for c, y in kids.items():
            lab[y] = c
    rd = np.zeros(V + 1, np.int32)
    rd[:V] = g.token_row(0)
    rp = g.psi32[rd].copy()
    rp[V] = 0.0
    return dict(first_child=fc, n_child=nc, link=np.asarray(g.link, np.int32), label=lab,
                phi=g.phi32, psi=g.psi32, root_dst=rd, root_psi=rp)


@pytest.mark.parametrize("tau,semantics,scale", [(1.0, COMMIT, None), (0.0, COMMIT, 0.75),
                                                 (2.0, PURE_POTENTIAL, None),
                                                 (0.5, COMMIT, 1.5)])
def test_compiler_matches_the_oracle(tau, semantics, scale):
    cfg = WP.piece_config("variative_small", B=5, n_phrases=25)
    toks = WP.vocab(cfg)
    lists = WP.phrases(cfg)
    lists[2] = []                                       # an empty list
    graphs = _compile(cfg, lists, toks, tau, scale=scale, semantics=semantics)
    img = graphs.host_image()
    L = graphs.layout
    capi.tb_validate_image(img, L)
    a = capi.image_arrays(img, L)
    assert np.array_equal(a["class_map"], oracle.class_map_of(toks, WP.LOWER))
    alpha = 1.0 if scale is None else scale
    for m, lst in enumerate(lists):
        g = oracle.build_variative_graph(toks, WP.LOWER, lst, token_w=cfg.token_w,
                                         end_bonus=cfg.end_bonus, alpha=alpha, tau=tau,
                                         semantics=semantics)
        f, n = int(a["model_off"][m]), int(a["model_n"][m])
        assert n == g.n_states, (m, n, g.n_states)
        want = _expected(g, cfg.V)
        for k in ("first_child", "n_child", "link", "label", "phi", "psi"):
            assert np.array_equal(a[k][f:f + n], want[k]), (m, k)
        assert np.array_equal(a["root_dst"][m], want["root_dst"]), m
        assert np.array_equal(a["root_psi"][m], want["root_psi"]), m


def test_every_character_needs_a_piece():
    cfg = WP.piece_config("variative_small", B=1, n_phrases=3)
    toks = [t for t in WP.vocab(cfg) if t != (5,) and t != (32,)]   # drop 'f' and 'F'
    bad = [[(26, 5, 0)]]
    with pytest.raises(capi.TbError) as e:
        _compile(cfg, bad, toks, 1.0)
    assert e.value.code == capi.TB_ERANGE


def test_argument_errors():
    cfg = WP.piece_config("variative_small", B=1, n_phrases=3)
    toks = WP.vocab(cfg)
    lists = WP.phrases(cfg)
    with pytest.raises(capi.TbError) as e:
        _compile(cfg, lists, toks, float("nan"))
    assert e.value.code == capi.TB_EINVAL
    with pytest.raises(capi.TbError) as e:
        _compile(cfg, [[()]], toks, 1.0)                               # an empty phrase
    assert e.value.code == capi.TB_ERANGE
    with pytest.raises(capi.TbError) as e:
        _compile(cfg, [[(26, 60)]], toks, 1.0)                          # character out of range
    assert e.value.code == capi.TB_ERANGE
    with pytest.raises(capi.TbError) as e:
        _compile(cfg, lists, toks[:10] + [()] + toks[11:], 1.0)         # a token without characters
    assert e.value.code == capi.TB_ERANGE
