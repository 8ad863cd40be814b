"""The pooled all-stream oracle used by the full-size GPU parity tests gives
exactly the outputs of the oracle run directly (CPU only)."""

import os

import numpy as np

import oracle
import workloads as W
from tests.gpu_cases import oracle_all_streams, oracle_graphs


def _spill(cfg, path):
    mm = np.lib.format.open_memmap(path, mode="w+",
                                   dtype=np.float32 if cfg.dtype == "f32" else np.uint16,
                                   shape=(cfg.T, cfg.B, cfg.K, cfg.Vp1))
    mm[:] = W.logits(cfg)
    mm.flush()
    del mm


def test_pooled_oracle_equals_direct_oracle(tmp_path):
    for name, over in (("batched", dict(T=60)), ("beam", dict(B=6, T=12))):
        cfg = W.config_by_name(name, **over)
        path = str(tmp_path / f"{name}.npy")
        _spill(cfg, path)
        pooled = oracle_all_streams(cfg, path, parts=4)
        lists = W.phrases(cfg)
        mids = W.model_ids(cfg)
        graphs = oracle_graphs(cfg, lists, range(cfg.B), mids)
        rows = W.logits(cfg)
        if cfg.K == 1:
            ref = oracle.greedy_decode(graphs, mids, rows, np.zeros(cfg.B, np.int32))
            n = 4
        else:
            st, S = oracle.init_carry(mids, cfg.K)
            ref = oracle.beam_decode(graphs, mids, rows, st, S)
            n = 5
        for i in range(n):
            assert np.array_equal(pooled[i], ref[i]), (name, i)
