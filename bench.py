"""Benchmark of the boosted decode step on one MI355X.

Default workload (the headline): streaming greedy decoding -- B=128 streams,
V=1024 tokens + blank, T=1024 steps fed as 64 calls of 16 steps each with the
graph states carried from call to call; fp32 joint logits N(0,1) with a +1.5
blank offset; every stream has its own list of 1000 phrases (lengths 1-10,
Zipf 1.1) and a case-insensitive token map. All inputs are synthetic and
seeded (workloads.logit_chunks) and are resident in HBM before the timed
region.

One bench step = one pass of the whole hot path over the workload: state
initialisation plus the workload's calls (64 calls of 16 steps for streaming,
one call of T steps for the others), states carried between calls. ``value``
is token-scores per second (T*B*K*(V+1) per step / step time). ``roofline``
describes the workload's step kernel: algorithmic bytes per launch over its
mean duration, from HIP events on the launch stream around each step's calls
in the timed region (their time over the number of calls, gaps between
launches included). For streaming, ``whole_call`` times the same workload
decoded by one call over all 1024 steps (the segmented kernel plus its
boundary fix-up), for context. ``read_probe`` times a plain read of the same
logit bytes, for context. Workloads whose logits are smaller than 512 MiB get
replicated buffers, one per bench step in turn, so that the last-level cache
does not hold a step's input. ``launch_floor_us`` is the mean time of an
empty kernel of the short-call kernel's shape launched the same number of
times through the same path: the part of a launch that is not the kernel's
work. For streaming, ``per_stream_vs_global`` times the same calls with every
stream on one model id (a single global tree) beside the per-stream lists.
``cpu_baseline`` times the CPU oracle over a
process pool on a bounded sample of the same workload (decode only), with a
single-process figure beside it.

Other workloads (--workload): batched, beam, stress_greedy, stress_beam, each
in its own launch pattern, for context; stress_beam prepares 4.3 GB of
logits on the host first (about two minutes). The default run also measures
batched, beam, stress_greedy and variative_streaming in short runs of their
own (child processes, 5 steps after 2 warm-up steps) and reports them under
``other_workloads`` (--no-others skips them).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
                       [--copy-probe] [--workload NAME] [--no-others]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
LAUNCH_FLOOR_LDS = 160 * 1024 - 1024
ROTATE_BYTES = 512 << 20
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "greedy_chunk_streaming_traffic.json")

KERNELS = {
    "streaming": "greedy short-call kernel (one launch per 16-step chunk)",
    "batched": "segmented greedy kernel + boundary fix-up (one call of 500 steps)",
    "beam": "beam kernel, one workgroup per stream (one call of 256 steps)",
    "stress_greedy": "wide-row greedy kernel, one workgroup per time segment, + boundary fix-up "
                     "(one call of 256 steps)",
    "stress_beam": "wide-row beam kernel, one workgroup per stream (one call of 256 steps)",
    "lifecycle": "greedy short-call kernel on a registry arena (one launch per 16-step chunk)",
    "variative_streaming": "greedy short-call kernel on variative BPE graphs (one launch per "
                           "16-step chunk)",
}

# CPU oracle sample per workload: (streams, steps); None = all
CPU_SAMPLE = {
    "streaming": (None, None),
    "batched": (None, None),
    "beam": (32, None),
    "stress_greedy": (64, 64),
    "stress_beam": (32, 16),
}


def _cpu_worker(args):
    """Oracle decode of some streams over steps [0, t1); returns (rows, seconds of decode)."""
    name, streams, t1 = args
    import oracle
    import workloads as W
    cfg = W.config_by_name(name)
    cm = W.class_map(cfg)
    lists = W.phrases(cfg, streams)
    graphs = {i: oracle.build_graph(l, cm, token_w=cfg.token_w, end_bonus=cfg.end_bonus)
              for i, l in enumerate(lists)}
    rows = W.logits(cfg, 0, t1, streams=streams)
    mids = list(range(len(streams)))
    t0 = time.perf_counter()
    if cfg.K == 1:
        oracle.greedy_decode(graphs, mids, rows, np.zeros(len(streams), np.int32))
    else:
        st, S = oracle.init_carry(mids, cfg.K)
        oracle.beam_decode(graphs, mids, rows, st, S)
    return rows.shape[0] * rows.shape[1] * rows.shape[2], time.perf_counter() - t0


def cpu_baseline(cfg):
    """The CPU oracle on a sample of the workload, one process per core."""
    import multiprocessing as mp
    n_streams, n_steps = CPU_SAMPLE[cfg.name]
    n_streams = cfg.B if n_streams is None else min(n_streams, cfg.B)
    t1 = cfg.T if n_steps is None else min(n_steps, cfg.T)
    cores = min(len(os.sched_getaffinity(0)), 16, n_streams)
    streams = list(range(n_streams))
    parts = [streams[i::cores] for i in range(cores)]
    ctx = mp.get_context("spawn")
    with ctx.Pool(cores) as pool:
        res = pool.map(_cpu_worker, [(cfg.name, p, t1) for p in parts if p])
    rows = sum(r for r, _ in res)
    secs = max(s for _, s in res)
    whole = n_streams == cfg.B and t1 == cfg.T
    what = "the whole workload" if whole else "a sample of the workload"
    # one process on the streams of the first part, for the single-core rate
    with ctx.Pool(1) as pool:
        rows1, secs1 = pool.map(_cpu_worker, [(cfg.name, parts[0], t1)])[0]
    return {
        "value": rows * cfg.Vp1 / secs,
        "unit": "token-scores/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"{what}: {n_streams} of {cfg.B} streams x {t1} of {cfg.T} steps "
                  f"({rows} rows of {cfg.Vp1} logits), streams split over {cores} processes; "
                  f"decode time only (graph building and logit generation untimed); "
                  f"wall = slowest process",
        "seconds": secs,
        "single_thread": {"value": rows1 * cfg.Vp1 / secs1, "seconds": secs1,
                          "sample": f"{len(parts[0])} streams x {t1} steps in one process"},
    }


def cache_levels(capi, W, cfg, cm, reg, spare, ws) -> dict:
    """Host wall time to give a stream a new model at each level of the model
    cache: compile its list, load it from a file, or take it from the
    host-memory cache, then copy it into the registry arena (each model is
    removed again afterwards); a model registered before the session only
    needs the stream's reset to its id. Mean over the spare lists."""
    import shutil
    import tempfile
    import torch
    cache = capi.GraphsCache(cm)
    tmp = tempfile.mkdtemp(prefix="tbias_models_")
    csrs = [W.phrase_csr([lst]) for lst in spare]  # the caller's lists, as the C-ABI takes them
    try:
        paths = []
        for j, csr in enumerate(csrs):
            g, _ = cache.compile(*csr, cfg.token_w, cfg.end_bonus)
            paths.append(os.path.join(tmp, f"model{j}.tbg"))
            capi.tb_graphs_save(g, paths[-1])

        def add_remove(make) -> float:
            torch.cuda.synchronize()
            t = time.perf_counter()
            new = reg.register(make())
            torch.cuda.synchronize()
            dt = time.perf_counter() - t
            reg.unregister(new[0], workspace=ws)
            torch.cuda.synchronize()
            return dt * 1e3

        out = {
            "compile": float(np.mean([add_remove(lambda: capi.tb_compile_graphs(
                *csr, cfg.token_w, cfg.end_bonus, cm)) for csr in csrs])),
            "disk": float(np.mean([add_remove(lambda: capi.tb_graphs_load(p)) for p in paths])),
            "memory": float(np.mean([add_remove(lambda: cache.compile(
                *csr, cfg.token_w, cfg.end_bonus)[0]) for csr in csrs])),
        }
        hits = cache.stats()["hits"]
        mids = torch.zeros(cfg.B, dtype=torch.int32, device="cuda")
        states = torch.zeros(cfg.B, dtype=torch.int32, device="cuda")
        walls = []
        for b in range(len(spare)):
            torch.cuda.synchronize()
            t = time.perf_counter()
            capi.tb_reset_stream(reg.arena, b, b, 1, mids, states)
            torch.cuda.synchronize()
            walls.append((time.perf_counter() - t) * 1e3)
        out["decoder"] = float(np.mean(walls))
        out["memory_hits"] = hits
        out["what"] = ("host wall ms per model: compile + copy into the arena; file load + copy; "
                       "host-memory cache hit + copy; registered before the session (the "
                       "stream's reset to its id)")
        return out
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


def lifecycle(args) -> int:
    """Model lifecycle next to the streaming step: the 128 streaming models in
    a registry arena (room for 8 more), then the cost of adding one compiled
    model (its records copied in, ids and offsets recorded) and of removing one
    from the middle (the later half of the arena moved left by the compaction
    kernel, the model table rebased), each as the mean of several, beside the
    streaming workload decoded through the registry arena."""
    import torch
    import workloads as W
    from paper_2608_21343_amd import capi
    from paper_2608_21343_amd.decoder import BoostDecoder

    cfg = W.config_by_name("streaming")
    T, B, V1, chunk = cfg.T, cfg.B, cfg.Vp1, cfg.chunk
    cm = W.class_map(cfg)
    lists = W.phrases(cfg)
    spare = W.phrases(W.config_by_name("streaming", B=B + 8), range(B, B + 8))
    t0 = time.perf_counter()
    g_all = capi.tb_compile_graphs(*W.phrase_csr(lists), cfg.token_w, cfg.end_bonus, cm)
    compile_s = time.perf_counter() - t0
    spare_g = [capi.tb_compile_graphs(*W.phrase_csr([l]), cfg.token_w, cfg.end_bonus, cm)
               for l in spare]
    cap = g_all.layout.n_states + sum(g.layout.n_states for g in spare_g)
    reg = capi.Registry(B + 8, cap, cm)
    ids = reg.register(g_all)
    stream = torch.cuda.current_stream()

    def timed(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t = time.perf_counter()
        a.record(stream)
        fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b), (time.perf_counter() - t) * 1e3

    add_ms, add_wall, rm_ms, rm_wall, moved = [], [], [], [], []
    ws = torch.empty(max(reg.workspace_bytes(i) for i in ids), dtype=torch.uint8, device="cuda")
    # untimed: the first launch of a kernel loads its code object (milliseconds)
    warm = reg.register(spare_g[0])
    reg.unregister(ids[len(ids) // 2], workspace=ws)
    reg.unregister(warm[0], workspace=ws)
    ids = ids[:len(ids) // 2] + ids[len(ids) // 2 + 1:] + reg.register(
        capi.tb_compile_graphs(*W.phrase_csr([lists[len(ids) // 2]]), cfg.token_w,
                               cfg.end_bonus, cm))
    for g in spare_g:
        new = []
        d, w = timed(lambda: new.extend(reg.register(g)))
        add_ms.append(d)
        add_wall.append(w)
        victim = ids[len(ids) // 2]
        moved.append(reg.workspace_bytes(victim))
        d, w = timed(lambda: reg.unregister(victim, workspace=ws))
        rm_ms.append(d)
        rm_wall.append(w)
        ids = [i for i in ids if i != victim] + new
    levels = cache_levels(capi, W, cfg, cm, reg, spare, ws)
    # the streaming workload through the registry arena (every stream on a live model)
    dec = BoostDecoder.for_arena(reg.arena)
    dt = torch.float32
    logits = torch.empty((T, B, V1), dtype=dt, device="cuda")
    for ta, tb, rows in W.logit_chunks(cfg, 16):
        logits[ta:tb].copy_(torch.from_numpy(rows[:, :, 0, :]).cuda())
    mids_np = np.asarray(sorted(ids)[:B], np.int32)
    mids, states, _ = dec.start(mids_np)
    outs = (torch.empty((T, B), dtype=torch.int32, device="cuda"),
            torch.empty((T, B), dtype=torch.int32, device="cuda"),
            torch.empty((T, B), dtype=torch.float32, device="cuda"))
    n_launch = T // chunk

    def run():
        capi.tb_init_states(dec.arena, B, 1, mids, states)
        for i in range(n_launch):
            ta, tb = i * chunk, (i + 1) * chunk
            capi.tb_boost_step_greedy(dec.arena, logits[ta:tb], mids, states,
                                      *(o[ta:tb] for o in outs))

    for _ in range(args.warmup):
        run()
    step_ms = [timed(run)[0] for _ in range(args.steps)]
    step_s = float(np.mean(step_ms)) / 1e3
    alg_bytes = chunk * B * (V1 * 4 + 12) + B * 12
    result = {
        "metric": "boosted decode token-scores/s (B x K x (V+1) per step) with achieved HBM GB/s",
        "value": T * B * V1 / step_s,
        "unit": "token-scores/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": step_s * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "lifecycle: streaming greedy decode (64 calls of 16 steps) on a "
                               "registry arena after 8 model additions and removals",
                   "B": B, "K": 1, "V": cfg.V, "T": T, "chunk": chunk,
                   "models": B, "spare_ids": 8, "arena_bytes": reg.arena.layout.total_bytes},
        "roofline": {"bound": "hbm", "achieved": alg_bytes / (step_s / n_launch) / 1e9,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": alg_bytes / (step_s / n_launch) / 1e9 / HBM_PEAK_GBS, "traffic": None,
                     "kernel": KERNELS["lifecycle"], "alg_bytes_per_launch": alg_bytes,
                     "avg_launch_us": step_s / n_launch * 1e6},
        "lifecycle": {
            "register_one_model_ms": float(np.mean(add_ms)),
            "register_one_model_wall_ms": float(np.mean(add_wall)),
            "unregister_one_model_ms": float(np.mean(rm_ms)),
            "unregister_one_model_wall_ms": float(np.mean(rm_wall)),
            "compaction_bytes_moved": int(np.mean(moved)),
            # the records are read and written twice (out to the workspace and back)
            "compaction_traffic_GBps": float(np.mean(moved)) * 4 / (float(np.mean(rm_ms)) / 1e3) / 1e9,
            "compile_128_models_s": compile_s,
            "step_ms": step_s * 1e3,
            "what": "one compiled model added (host records copied in, table updated, "
                    "synchronised) and one model removed from the middle of 128 (the later "
                    "records moved left through a workspace, table rebased on the device), "
                    "device time between events and host wall time, mean of 8 each",
            "add_one_model_by_cache_level_ms": levels,
            "per_16_step_call_ms": step_s * 1e3 / n_launch,
        },
    }
    print(json.dumps(result), flush=True)
    return 0


def stream_beam_figures(dec, cfg, rows_dev, mids, stream, reps: int = 4) -> dict:
    """The beam workload through the streaming beam (recombination and a
    flattened tree of 4096 records per stream): one call over all steps, and
    the steps as calls of 16, eager and as one captured HIP graph of the
    whole chunk loop."""
    import torch
    from paper_2608_21343_amd import capi
    T, B, K = cfg.T, cfg.B, cfg.K
    chunk = 16
    i32 = dict(dtype=torch.int32, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    outs = tuple(torch.empty((T, B, K), **i32) for _ in range(3)) + \
        tuple(torch.empty((T, B, K), **f32) for _ in range(2))
    carry = dec.start_beam_stream(mids, K, 4096)

    def restart():
        capi.tb_init_beam_stream(dec.arena, B, K, carry.mids, carry.states, carry.scores,
                                 carry.hyps, carry.tree_len)

    def timed(body):
        ms = []
        for rep in range(reps + 1):
            restart()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            body()
            b.record(stream)
            torch.cuda.synchronize()
            if rep > 0:
                ms.append(a.elapsed_time(b))
        return float(np.mean(ms))

    one_ms = timed(lambda: dec.beam_stream(rows_dev, carry, out=outs))
    whole = tuple(o.clone() for o in outs)
    n = T // chunk

    def chunks():
        for i in range(n):
            dec.beam_stream(rows_dev[i * chunk:(i + 1) * chunk], carry,
                            out=tuple(o[i * chunk:(i + 1) * chunk] for o in outs))

    eager_ms = timed(chunks)
    same = all(torch.equal(x, y) for x, y in zip(whole, outs))
    # the chunk loop captured once as a HIP graph (every call on its own
    # slices of the resident rows) and replayed per step
    restart()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        chunks()
    graph_ms = timed(g.replay)
    same_graph = all(torch.equal(x, y) for x, y in zip(whole, outs))
    m2, st, sc = dec.start(mids, K)

    def plain():
        capi.tb_init_states(dec.arena, B, K, m2, st, sc)
        dec.beam(rows_dev, m2, st, sc, out=outs)

    plain_ms = timed(plain)
    del g
    return {"one_call_ms": one_ms, "plain_beam_one_call_ms": plain_ms,
            "recombination_cost": one_ms / plain_ms,
            "calls_of_16_eager_ms": eager_ms, "calls_of_16_graph_ms": graph_ms,
            "chunked_equals_one_call": bool(same), "graph_equals_one_call": bool(same_graph),
            "tree_cap": 4096}


# Workloads the default run also measures, each in a child process with a
# short run of its own (the stress beam's 4.3 GB of host-side logits take too
# long for the default run).
OTHER_WORKLOADS = ("batched", "beam", "stress_greedy", "variative_streaming")


def other_workloads(steps: int, warmup: int) -> dict:
    """Short bench runs of the other workloads (child processes, one at a
    time): per workload its step time, throughput and roofline figures."""
    import subprocess
    out = {}
    for w in OTHER_WORKLOADS:
        print(f"bench: workload {w}", file=sys.stderr, flush=True)
        t0 = time.perf_counter()
        cmd = [sys.executable, os.path.abspath(__file__), "--workload", w, "--steps", str(steps),
               "--warmup", str(warmup), "--no-cpu-baseline", "--no-others"]
        try:
            p = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
        except subprocess.TimeoutExpired:
            out[w] = {"error": "timed out after 300 s"}
            continue
        lines = [ln for ln in p.stdout.splitlines() if ln.startswith("{")]
        if p.returncode != 0 or not lines:
            out[w] = {"error": f"exit {p.returncode}: {p.stderr.strip()[-300:]}"}
            continue
        d = json.loads(lines[-1])
        r = d["roofline"]
        out[w] = {"workload": d["config"]["workload"], "ms_per_step": d["ms_per_step"],
                  "value": d["value"], "unit": d["unit"], "dtype": d["dtype"],
                  "avg_launch_us": r["avg_launch_us"], "achieved_GBps": r["achieved"],
                  "frac": r["frac"], "kernel": r["kernel"], "steps": d["steps"],
                  "run_s": time.perf_counter() - t0}
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="first run one plain 256 MiB device copy (counter calibration)")
    ap.add_argument("--workload", default="streaming", choices=sorted(KERNELS))
    ap.add_argument("--no-others", action="store_true",
                    help="streaming only: skip the short runs of the other workloads")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the streams "
              f"are independent: more GPUs would each run their own share of the streams with "
              f"no exchange between steps)", file=sys.stderr)
        return 2

    import torch
    import workloads as W
    from paper_2608_21343_amd import capi, profiling
    from paper_2608_21343_amd.decoder import BoostDecoder

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    if args.copy_probe:
        n = profiling.COPY_PROBE_BYTES // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    if args.workload == "lifecycle":
        return lifecycle(args)
    variative = args.workload.startswith("variative")
    if variative:
        import workloads.pieces as WP
        cfg = WP.piece_config(args.workload)
        args.no_cpu_baseline = True   # the oracle's variative compile is far too slow here
    else:
        cfg = W.config_by_name(args.workload)
    T, B, K, V1, chunk = cfg.T, cfg.B, cfg.K, cfg.Vp1, cfg.chunk
    item = 4 if cfg.dtype == "f32" else 2
    if variative:
        pieces = WP.vocab(cfg)
        lists = WP.phrases(cfg)
        t0 = time.perf_counter()
        dec = BoostDecoder.variative(lists, pieces, WP.LOWER, cfg.tau, token_w=cfg.token_w,
                                     end_bonus=cfg.end_bonus)
        compile_s = time.perf_counter() - t0
        plant_map = {}
        for b, lst in enumerate(lists):
            for t, v in WP.plants(cfg, b, pieces, lst):
                plant_map.setdefault(t, []).append((b, v))
        chunks_src = WP.logit_chunks(cfg, 16, plant_map=plant_map)
    else:
        lists = W.phrases(cfg)
        t0 = time.perf_counter()
        dec = BoostDecoder(lists, W.class_map(cfg), token_w=cfg.token_w, end_bonus=cfg.end_bonus)
        compile_s = time.perf_counter() - t0
        chunks_src = W.logit_chunks(cfg, 16)
    dt = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
    logits = torch.empty((T, B, K, V1), dtype=dt, device="cuda")
    t0 = time.perf_counter()
    for ta, tb, rows in chunks_src:
        h = torch.from_numpy(rows if cfg.dtype == "f32" else rows.view(np.int16))
        logits[ta:tb].copy_(h.cuda().view(dt))
        del h, rows
        if time.perf_counter() - t0 > 20:  # progress of long preparations (stderr)
            print(f"bench: logits up to step {tb} of {T} on the device", file=sys.stderr, flush=True)
            t0 = time.perf_counter()
    # Logits smaller than the 256 MB last-level cache are replicated so that
    # consecutive bench steps read different buffers (at least 512 MiB apart).
    n_buf = max(1, -(-ROTATE_BYTES // (logits.numel() * item)))
    bufs = [logits] + [logits.clone() for _ in range(n_buf - 1)]
    mids, states, scores = dec.start(np.arange(B, dtype=np.int32), K)
    i32 = dict(dtype=torch.int32, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    if K == 1:
        rows_bufs = [x[:, :, 0, :] for x in bufs]
        outs = (torch.empty((T, B), **i32), torch.empty((T, B), **i32),
                torch.empty((T, B), **f32))
    else:
        rows_bufs = bufs
        outs = tuple(torch.empty((T, B, K), **i32) for _ in range(3)) + \
            tuple(torch.empty((T, B, K), **f32) for _ in range(2))
    n_launch = (T + chunk - 1) // chunk
    stream = torch.cuda.current_stream()

    def call(ta, tb, rows_dev):
        sl = tuple(o[ta:tb] for o in outs)
        if K == 1:
            capi.tb_boost_step_greedy(dec.arena, rows_dev[ta:tb], mids, states, *sl)
        else:
            capi.tb_boost_step_beam(dec.arena, rows_dev[ta:tb], mids, states, scores, *sl)

    n_run = [0]

    def run_step(events=None):
        rows_dev = rows_bufs[n_run[0] % n_buf]
        n_run[0] += 1
        capi.tb_init_states(dec.arena, B, K, mids, states, scores)
        if events is not None:
            events[0].record(stream)
        for i in range(n_launch):
            ta, tb = i * chunk, min(T, (i + 1) * chunk)
            call(ta, tb, rows_dev)
        if events is not None:
            events[1].record(stream)

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()
    # one event pair per step around its calls: events between the calls of a
    # step would add their own cost to the timed region (about a fifth of the
    # streaming step), so the mean launch time is the bracketed calls over
    # their number, gaps between launches included
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        run_step(ev[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    launch_ms = [a.elapsed_time(b) / n_launch for (a, b) in ev]
    avg_launch_s = float(np.mean(launch_ms)) / 1e3
    kept = tuple(o.clone() for o in outs)

    step_s = wall / args.steps
    token_scores = T * B * K * V1
    # algorithmic bytes per launch: the call's logit rows read once, the
    # outputs of every row (token, state, score; beam also parent and
    # cumulative score), and per stream the model id plus the carried states
    # (and beam scores) read and written
    out_b = 12 if K == 1 else 20
    carry_b = 4 + K * (8 if K == 1 else 16)
    alg_bytes = chunk * B * K * (V1 * item + out_b) + B * carry_b
    achieved = alg_bytes / avg_launch_s / 1e9

    result = {
        "metric": "boosted decode token-scores/s (B x K x (V+1) per step) with achieved HBM GB/s",
        "value": token_scores / step_s,
        "unit": "token-scores/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {'greedy' if K == 1 else f'beam K={K}'} boosted decode, "
                               f"{n_launch} call{'s' if n_launch > 1 else ''} of {chunk} steps",
                   "B": B, "K": K, "V": cfg.V, "T": T, "chunk": chunk,
                   "logits": f"{cfg.dtype} N(0,{cfg.logit_std:g})"
                             + (f", blank +{cfg.blank_offset:g}" if cfg.blank_offset else ""),
                   "phrases_per_stream": cfg.n_phrases, "launches_per_step": n_launch},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS,
                     "traffic": (profiling.load_traffic(TRAFFIC_FILE)
                                 if cfg.name == "streaming" else None),
                     "kernel": KERNELS[cfg.name],
                     "alg_bytes_per_launch": alg_bytes, "avg_launch_us": avg_launch_s * 1e6},
        "steps_per_s": T / step_s,
        "compile_s": compile_s,
        "rotated_buffers": n_buf,
    }

    # context: a plain read of the same logit bytes (torch's max reduction)
    probe_ms = []
    for rep in range(4):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        x = bufs[rep % n_buf]
        a.record(stream)
        torch.amax(x)
        b.record(stream)
        torch.cuda.synchronize()
        if rep > 0:
            probe_ms.append(a.elapsed_time(b))
    probe_s = float(np.median(probe_ms)) / 1e3
    result["read_probe"] = {"GBps": logits.numel() * item / probe_s / 1e9,
                            "bytes": logits.numel() * item,
                            "what": "torch.amax over the workload's logits, median of 3"}

    # the launch floor: an empty kernel of the short-call kernel's shape (one
    # workgroup of 16 waves per stream, its LDS), launched as often as the
    # step's calls through the same path, one event pair around them
    floor_ms = []
    for rep in range(4):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(n_launch):
            capi.tb_debug_launch_empty(B, 1024, LAUNCH_FLOOR_LDS)
        b.record(stream)
        torch.cuda.synchronize()
        if rep > 0:
            floor_ms.append(a.elapsed_time(b) / n_launch)
    result["launch_floor_us"] = float(np.median(floor_ms)) * 1e3
    result["launch_floor_shape"] = f"{B} workgroups x 1024 threads, {LAUNCH_FLOOR_LDS} B LDS"

    if cfg.name == "streaming":
        # every stream on one model id (a single global tree) against the
        # per-stream lists above: the same calls, states carried, timed the
        # same way (the paper reports no observable speed difference)
        gdec = BoostDecoder([lists[0]], W.class_map(cfg), token_w=cfg.token_w,
                            end_bonus=cfg.end_bonus)
        gm, gst, gsc = gdec.start(np.zeros(B, np.int32), K)
        g_ms = []
        for rep in range(args.steps + 1):
            rows_dev = rows_bufs[rep % n_buf]
            capi.tb_init_states(gdec.arena, B, K, gm, gst, gsc)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for i in range(n_launch):
                ta, tb = i * chunk, min(T, (i + 1) * chunk)
                capi.tb_boost_step_greedy(gdec.arena, rows_dev[ta:tb], gm, gst,
                                          *(o[ta:tb] for o in outs))
            b.record(stream)
            torch.cuda.synchronize()
            if rep > 0:
                g_ms.append(a.elapsed_time(b))
        per_ms = float(np.mean([a.elapsed_time(b) for (a, b) in ev]))
        glob_ms = float(np.mean(g_ms))
        result["per_stream_vs_global"] = {
            "per_stream_ms": per_ms, "global_ms": glob_ms,
            "per_stream_token_scores_per_s": token_scores / (per_ms / 1e3),
            "global_token_scores_per_s": token_scores / (glob_ms / 1e3),
            "ratio": per_ms / glob_ms,
            "what": f"the step's {n_launch} calls: {B} streams with their own lists (model b) "
                    f"against all {B} streams on one model id (stream 0's list)"}
        del gdec

    if cfg.name == "streaming":
        # context: the same workload as one call over all T steps
        whole_ms = []
        for rep in range(4):
            capi.tb_init_states(dec.arena, B, 1, mids, states)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            call(0, T, rows_bufs[0])
            b.record(stream)
            torch.cuda.synchronize()
            if rep > 0:
                whole_ms.append(a.elapsed_time(b))
        whole_s = float(np.median(whole_ms)) / 1e3
        whole_bytes = T * B * (V1 * item + out_b) + B * carry_b
        same = all(torch.equal(x, y) for x, y in zip(kept[:2], outs[:2]))
        result["whole_call"] = {"ms": whole_s * 1e3, "token_scores_per_s": token_scores / whole_s,
                                "achieved_GBps": whole_bytes / whole_s / 1e9,
                                "frac": whole_bytes / whole_s / 1e9 / HBM_PEAK_GBS,
                                "kernels": "segmented greedy kernel + boundary fix-up",
                                "outputs_equal_chunked": bool(same)}
    if variative:
        L = dec.arena.layout
        result["variative"] = {
            "pieces": cfg.V, "tau": cfg.tau, "states": int(L.n_states),
            "states_per_list": int(L.n_states) / B, "arena_MB": L.total_bytes / 1e6,
            "max_override": int(L.max_override), "compile_s": compile_s,
            "what": "lists written in characters over a synthetic piece vocabulary, one state "
                    "per arc of the variative graph; phrases planted as random segmentations "
                    "and casings every 16 steps"}
    if cfg.name == "beam":
        result["stream_beam"] = stream_beam_figures(dec, cfg, rows_bufs[0], W.model_ids(cfg),
                                                    stream)
    del logits, bufs, rows_bufs
    if cfg.name == "streaming" and not args.no_others:
        torch.cuda.empty_cache()
        result["other_workloads"] = other_workloads(steps=5, warmup=2)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
