"""Decodes through the LDS-poisoning debug build, against the oracle (run by
tests/test_gpu_poison.py in a child process).

argv[1] is a directory holding a copy of the package whose library is the
poison build; it goes first on sys.path. Every kernel family runs once on a
small case: greedy short-call, segmented with fix-up, wide-row and reference
kernels; beam one-wave-per-hypothesis (with its row preparation), helper-wave,
wide-row and reference kernels; the streaming beam on the fast and the
reference kernel; a variative graph."""

import os
import sys

sys.path.insert(0, sys.argv[1])
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(1, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import workloads as W  # noqa: E402
import workloads.pieces as WP  # noqa: E402
from paper_2608_21343_amd import capi  # noqa: E402
from paper_2608_21343_amd.decoder import BoostDecoder, to_device_logits  # noqa: E402
from tests.gpu_cases import compare_beam, compare_greedy, gpu_beam, gpu_greedy  # noqa: E402

assert os.path.dirname(str(capi.LIB_PATH)).startswith(sys.argv[1]), capi.LIB_PATH


def case(V, K, T, dtype="f32", B=6, seed=0):
    cfg = W.Config(900 + seed, "poison", B=B, K=K, V=V, T=T, chunk=16, dtype=dtype,
                   n_phrases=60, len_lo=1, len_hi=6, token_dist="zipf", zipf_s=1.1,
                   logit_std=1.0, blank_offset=1.0, n_case=max(1, V // 9))
    lists = W.phrases(cfg)
    dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
    mids = np.arange(B, dtype=np.int32)
    mids[1] = -1
    graphs = {int(m): oracle.build_graph(lists[int(m)], W.class_map(cfg), token_w=cfg.token_w,
                                         end_bonus=cfg.end_bonus) for m in mids if m >= 0}
    return cfg, dec, mids, graphs, W.logits(cfg)


def greedy(V, T, chunk, dtype="f32", kernel=capi.GREEDY_AUTO):
    capi.tb_debug_select_kernels(greedy=kernel)
    cfg, dec, mids, graphs, rows = case(V, 1, T, dtype, seed=V + T)
    gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, chunk)
    st0 = np.where(mids >= 0, 0, -1).astype(np.int32)
    compare_greedy(gpu, oracle.greedy_decode(graphs, mids, rows[:, :, 0, :], st0),
                   range(cfg.B), 1e-5)
    print(f"greedy V={V} T={T} chunk={chunk} {dtype} kernel={kernel}: ok", flush=True)


def beam(V, K, T, dtype="f32", kernel=capi.BEAM_AUTO):
    capi.tb_debug_select_kernels(beam=kernel)
    cfg, dec, mids, graphs, rows = case(V, K, T, dtype, seed=V + K)
    gpu = gpu_beam(dec, to_device_logits(rows), mids, 16)
    st0, S0 = oracle.init_carry(mids, K)
    compare_beam(gpu, oracle.beam_decode(graphs, mids, rows, st0, S0), range(cfg.B), 1e-5)
    print(f"beam V={V} K={K} {dtype} kernel={kernel}: ok", flush=True)


def stream_beam(V, K, T, kernel=capi.BEAM_AUTO):
    capi.tb_debug_select_kernels(beam=kernel)
    cfg, dec, mids, graphs, rows = case(V, K, T, seed=2 * V + K)
    rows_dev = to_device_logits(rows)
    carry = dec.start_beam_stream(mids, K, 512)
    ref = oracle.init_stream_carry(mids, K)
    for t0 in range(0, T, 16):
        gpu = [o.cpu().numpy() for o in dec.beam_stream(rows_dev[t0:t0 + 16], carry)]
        want = oracle.beam_decode_stream(graphs, mids, rows[t0:t0 + 16], ref, tree_cap=512)
        compare_beam(gpu, want, range(cfg.B), 1e-5)
    print(f"stream beam V={V} K={K} kernel={kernel}: ok", flush=True)


def variative():
    cfg = WP.piece_config("variative_small", index=77, B=6, T=48)
    toks, lists, rows = WP.vocab(cfg), WP.phrases(cfg), WP.logits(cfg)
    dec = BoostDecoder.variative(lists, toks, WP.LOWER, cfg.tau)
    mids = np.arange(cfg.B, dtype=np.int32)
    graphs = {int(m): oracle.build_variative_graph(toks, WP.LOWER, lists[int(m)], tau=cfg.tau)
              for m in mids}
    gpu = gpu_greedy(dec, to_device_logits(rows[:, :, 0, :]), mids, 16)
    compare_greedy(gpu, oracle.greedy_decode(graphs, mids, rows[:, :, 0, :],
                                             np.zeros(cfg.B, np.int32)), range(cfg.B), 1e-5)
    print("variative greedy: ok", flush=True)


greedy(300, 48, 16)                                   # short-call kernel
greedy(300, 200, 200)                                 # segmented kernel + fix-up
greedy(3000, 96, 96, "bf16")                          # wide-row kernel
greedy(300, 48, 16, kernel=capi.GREEDY_REF)           # reference kernel
beam(300, 8, 40)                                      # row preparation + one wave per hypothesis
beam(3000, 4, 24, "bf16")                             # helper waves
beam(3000, 8, 24, kernel=capi.BEAM_NO_PIPE)           # wide-row kernel
beam(300, 5, 24, kernel=capi.BEAM_REF)                # reference kernel
stream_beam(300, 8, 32)                               # streaming stage, fast kernel
stream_beam(300, 4, 32, kernel=capi.BEAM_REF)         # streaming stage, reference kernel
capi.tb_debug_select_kernels(capi.GREEDY_AUTO, capi.BEAM_AUTO)
variative()
print("poison checks: ok", flush=True)
