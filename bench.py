#!/usr/bin/env python3
"""Benchmark one batched paged-KV decode-attention step on one MI355X.

A "step" is one call of the library's decode attention (the stream-K decode
kernel plus the log-sum-exp combine kernel) over one synthetic decode batch
whose inputs are already resident in HBM. ``--op append`` times the KV append
of a decode step instead, and ``--op prefill`` the causal varlen prefill of a
log-prob forward (plan kernel plus attention kernel, MFMA-bound: reported in
TFLOP/s of the causal QK^T and PV products). Default workload: the largest
decode step that fits one GPU, fp8 KV at scale (512 sequences, 64 query / 8 KV
heads, head_dim 128, e4m3 cache with per-tile scales, lognormal lengths with
median 8192 up to 65,536); the same line then times the other long-tailed GQA
steps (7B GQA, GRPO rollout batch, stragglers) under ``per_config``. Smaller
caches are rotated over enough copies that consecutive steps never find their
cache in the 256 MB last-level cache.

Prints one JSON line. `value` is achieved GB/s of algorithmic bytes (K/V
tiles of every token, fp8 scales, q, out, block-table entries, lengths) over
the wall-clock step time; `roofline.achieved` is the same bytes over the
average per-call GPU time measured with HIP events on the launch stream.
`cpu_baseline` times the CPU fp64 oracle on a bounded sample of the same step.
"""

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFS = 2500.0   # dense bf16 matrix-core peak of MI355X
LLC_BYTES = 256 << 20
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2605_20863_amd", "csrc", "pda_kernels.hip")
PREFILL_SOURCE = os.path.join(ROOT, "paper_2605_20863_amd", "csrc", "pda_prefill.hip")


def algorithmic_bytes(workload, seq_lens, shared=None):
    """Bytes one step must move at least: each token's K and V once, plus
    fp8 scales, q, out, block-table entries and lengths. With ``shared`` =
    (group_size, shared_blocks) the blocks a group's members share count once
    (the unique bytes of a GRPO step); the token count stays the logical one."""
    e_kv = {"f32": 4, "bf16": 2, "fp8_e4m3": 1}[workload.kv_dtype]
    e_q = 4 if workload.q_dtype == "f32" else 2
    tokens = int(seq_lens.sum())
    blocks = int(((seq_lens.astype("int64") + 15) // 16).sum())
    B, hq, hkv, d = len(seq_lens), workload.num_q_heads, workload.num_kv_heads, workload.head_dim
    kv_tokens, kv_blocks = tokens, blocks
    if shared is not None:
        gs, sb = shared
        dup = int((gs - 1) * sb.astype("int64").sum())   # shared blocks beyond one copy per group
        kv_tokens -= 16 * dup
        kv_blocks -= dup
    kv = kv_tokens * hkv * 2 * d * e_kv
    scales = kv_blocks * hkv * 2 * 4 if workload.kv_dtype == "fp8_e4m3" else 0
    return kv + scales + 2 * B * workload.q_tokens * hq * d * e_q + 4 * blocks + 4 * B, tokens


def append_bytes(workload, B):
    """Bytes one KV append of a decode step must move: every sequence's new K
    and V rows read (bf16) and written in the cache dtype, fp8 tile scales read
    and written, positions and block-table entries. Re-encoding a tile whose
    scale grows is data-dependent and not counted."""
    e_kv = {"f32": 4, "bf16": 2, "fp8_e4m3": 1}[workload.kv_dtype]
    hkv, d = workload.num_kv_heads, workload.head_dim
    scales = 2 * 2 * B * hkv * 4 if workload.kv_dtype == "fp8_e4m3" else 0
    return 2 * B * hkv * d * (2 + e_kv) + scales + 8 * B


def prefill_flops(workload, seq_lens, counts):
    """Multiply-add flops of a causal prefill: query i of sequence b sees
    min(max(L - n + i + 1, 0), L) keys, and each visible (query head, key) pair
    costs D multiply-adds in QK^T and D in PV (2 flops each)."""
    import numpy as np

    pairs = 0
    for L, n in zip(seq_lens.astype(np.int64), counts.astype(np.int64)):
        vis = np.clip(L - n + np.arange(1, n + 1), 0, L)
        pairs += int(vis.sum())
    return 4 * workload.head_dim * workload.num_q_heads * pairs, pairs


# ----------------------------------------------------------------- CPU baseline

# Host cores that the process driving one MI355X may use: one GPU's share of
# an 8-GPU host's cores, whatever the affinity mask shows; more workers would
# only oversubscribe them.
CPU_SHARE = 16


def _worker_init():
    # one BLAS thread per oracle process (the pool already uses every core)
    for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[k] = "1"


def _pool_cores():
    """(cores the affinity mask shows, worker processes used)."""
    avail = len(os.sched_getaffinity(0))
    return avail, min(avail, CPU_SHARE)


def _cores_note(avail, used):
    if used < avail:
        return (f"{used} of the {avail} cores in the affinity mask: one GPU's share of the host is "
                f"{CPU_SHARE} cores")
    return f"all {avail} cores in the affinity mask"


def _close_pool(pool):
    """Terminate the oracle workers and wait for them to exit."""
    pool.terminate()
    pool.join()


def _stop_semaphore_tracker():
    """Wait for the semaphore tracker process that the spawn start method
    runs, once every pool (and so every semaphore) is gone, so that no process
    outlives the bench."""
    import gc

    gc.collect()
    try:
        from multiprocessing import resource_tracker
        resource_tracker._resource_tracker._stop()
    except Exception:  # private API; a leftover tracker exits with its parent
        pass


def _oracle_one(args):
    import oracle  # the CPU fp64 reference; test infrastructure

    (q, kc, vc, table, lens, scale, q_dtype, kv_dtype, ks) = args
    t0 = time.perf_counter()
    oracle.paged_decode_attention(q=q, k_cache=kc, v_cache=vc, block_table=table, seq_lens=lens,
                                  softmax_scale=scale, q_dtype=q_dtype, kv_dtype=kv_dtype, kv_scales=ks)
    return time.perf_counter() - t0


def _sequence_problem(inp, b, raw):
    """Host copy of sequence b's blocks as a one-sequence problem (data movement only)."""
    import numpy as np
    import torch

    lay = inp.layout
    n = (int(lay.seq_lens[b]) + 15) // 16
    phys = lay.block_table[b, :max(n, 1)].astype(np.int64)
    if n == 0:
        phys = np.zeros(1, dtype=np.int64)
    idx = torch.from_numpy(phys).to(inp.device)
    kc = raw(inp.k_cache.index_select(0, idx))
    vc = raw(inp.v_cache.index_select(0, idx))
    ks = raw(inp.kv_scales.index_select(1, idx)) if inp.kv_scales is not None else None
    table = np.arange(max(n, 1), dtype=np.int32)[None, :]
    w = inp.workload
    return (raw(inp.q[b:b + 1]), kc, vc, table, lay.seq_lens[b:b + 1].copy(), inp.softmax_scale,
            w.q_dtype, w.kv_dtype, ks)


def _oracle_prefill_rows(args):
    import oracle  # the CPU fp64 reference; test infrastructure

    t0 = time.perf_counter()
    oracle.paged_prefill_attention(**args)
    return time.perf_counter() - t0


def _prefill_rows_problem(pin, b, rows, raw):
    """Query rows ``rows`` of sequence b as one-token prefills over its cache cut
    at each row's position (a causal query sees nothing past it); host copies of
    the blocks they need (data movement only)."""
    import numpy as np
    import torch

    c = pin.cache
    L, n = int(c.layout.seq_lens[b]), int(pin.counts[b])
    pos = np.array([L - n + int(i) for i in rows], dtype=np.int64)
    nb = int(pos.max()) // 16 + 1
    idx = torch.from_numpy(c.layout.block_table[b, :nb].astype(np.int64)).to(c.device)
    w = c.workload
    qrows = torch.tensor([int(pin.offsets[b]) + int(i) for i in rows], dtype=torch.long, device=c.device)
    return dict(q=raw(pin.q.index_select(0, qrows)), q_offsets=np.arange(len(rows) + 1, dtype=np.int32),
                k_cache=raw(c.k_cache.index_select(0, idx)), v_cache=raw(c.v_cache.index_select(0, idx)),
                block_table=np.tile(np.arange(nb, dtype=np.int32), (len(rows), 1)),
                seq_lens=(pos + 1).astype(np.int32), softmax_scale=c.softmax_scale, q_dtype="bf16",
                kv_dtype=w.kv_dtype,
                kv_scales=raw(c.kv_scales.index_select(1, idx)) if c.kv_scales is not None else None), pos


def cpu_baseline_prefill(pin, budget_s, rows_per_job=4):
    """Time the oracle on seeded query rows of the prefill, one worker process
    per host core of one GPU's share."""
    import multiprocessing as mp

    import numpy as np
    import torch

    def raw(t):
        t = t.detach().cpu().contiguous()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.numpy()

    w = pin.cache.workload
    avail, cores = _pool_cores()
    rng = np.random.default_rng(0)
    seq_of_row = np.repeat(np.arange(len(pin.counts)), pin.counts)
    ctx = mp.get_context("spawn")
    pairs, nrows, t_cpu = 0, 0, 0.0
    pool = ctx.Pool(cores, initializer=_worker_init)
    try:
        t0 = time.perf_counter()
        pending = []
        while True:
            r = int(rng.integers(0, len(seq_of_row)))
            b = int(seq_of_row[r])
            i0 = r - int(pin.offsets[b])
            rows = list(range(i0, min(i0 + rows_per_job, int(pin.counts[b]))))
            job, pos = _prefill_rows_problem(pin, b, rows, raw)
            pending.append((int((pos + 1).sum()), len(rows), pool.apply_async(_oracle_prefill_rows, (job,))))
            if len(pending) >= 2 * cores:
                pp, nr, res = pending.pop(0)
                t_cpu += res.get()
                pairs, nrows = pairs + pp, nrows + nr
                if time.perf_counter() - t0 > budget_s:
                    break
        for pp, nr, res in pending:
            t_cpu += res.get()
            pairs, nrows = pairs + pp, nrows + nr
        wall = time.perf_counter() - t0
    finally:
        _close_pool(pool)
    flops = 4 * w.head_dim * w.num_q_heads * pairs
    return {
        "value": round(flops / wall / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": cores,
        "cores_available": avail,
        "cores_note": _cores_note(avail, cores),
        "kind": "oracle",
        "tokens_per_s": round(nrows / wall, 2),
        "seconds": round(wall, 2),
        "cpu_seconds": round(t_cpu, 2),
        "sample": f"{nrows} query rows (all {w.num_q_heads} heads; runs of {rows_per_job} consecutive rows from "
                  f"seeded positions) of the same prefill, {pairs} visible (row, key) pairs, fp64 numpy oracle, "
                  f"one process per core",
    }


def cpu_baseline(inp, budget_s):
    """Time the oracle over a seeded sample of sequences, one worker process
    per host core of one GPU's share."""
    import multiprocessing as mp

    import numpy as np
    import torch

    def raw(t):
        t = t.detach().cpu().contiguous()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.numpy()

    avail, cores = _pool_cores()
    lay = inp.layout
    order = np.random.default_rng(0).permutation(len(lay.seq_lens))
    ctx = mp.get_context("spawn")
    done, t_cpu = [], 0.0
    pool = ctx.Pool(cores, initializer=_worker_init)
    try:
        t0 = time.perf_counter()
        pending = []
        # keep the pool fed, pass after pass over the step's sequences, until the
        # wall budget is spent; every submitted sequence is finished and counted
        stop = False
        while not stop:
            for b in order:
                pending.append((int(b), pool.apply_async(_oracle_one, (_sequence_problem(inp, int(b), raw),))))
                if len(pending) >= 2 * cores:
                    bb, r = pending.pop(0)
                    t_cpu += r.get()
                    done.append(bb)
                    if time.perf_counter() - t0 > budget_s:
                        stop = True
                        break
            if time.perf_counter() - t0 > budget_s:
                stop = True
        for bb, r in pending:
            t_cpu += r.get()
            done.append(bb)
        wall = time.perf_counter() - t0
    finally:
        _close_pool(pool)
    lens = lay.seq_lens[done]
    nbytes, tokens = algorithmic_bytes(inp.workload, lens)
    return {
        "value": round(nbytes / wall / 1e9, 4),
        "unit": "GB/s",
        "cores": cores,
        "cores_available": avail,
        "cores_note": _cores_note(avail, cores),
        "kind": "oracle",
        "kv_tokens_per_s": round(tokens / wall, 1),
        "seconds": round(wall, 2),
        "cpu_seconds": round(t_cpu, 2),
        "sample": f"{len(done)} sequence evaluations ({tokens} tokens) of the same step, its "
                  f"{len(lay.seq_lens)} sequences taken in a seeded order (again from the start if the budget "
                  f"outlasts them), fp64 numpy oracle, one process per core",
    }


# ----------------------------------------------------------------- traffic

def source_digest(path):
    """sha256 of a kernel source's code: comments removed and whitespace
    collapsed, so that editing a comment keeps measurements taken on the same
    code valid, while any change to the code itself invalidates them."""
    import re

    text = open(path, encoding="utf-8").read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    text = " ".join(text.split())
    return hashlib.sha256(text.encode()).hexdigest()


def per_call_spread(step, n, stream, first):
    """GPU time of each of n more calls (us), every call between two HIP events
    on the calls' stream, run after the timed region: events between calls add
    their own GPU time, so this gives the spread (median, min, max) and the
    headline figure stays the one of the timed region."""
    import torch
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for i in range(n):
        step(first + i)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    t = sorted(evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(n))
    med = t[n // 2] if n % 2 else 0.5 * (t[n // 2 - 1] + t[n // 2])
    return {"median": round(med, 2), "min": round(t[0], 2), "max": round(t[-1], 2), "calls": n}


def measured_traffic(workload_name, per_launch_bytes, source=KERNEL_SOURCE):
    """HBM bytes per call from committed rocprofv3 FETCH_SIZE / WRITE_SIZE runs,
    or None when absent or taken on different kernel code."""
    path = os.path.join(PROFILES, f"traffic_{workload_name}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_code_sha256") != source_digest(source):
        return None
    return rec.get("hbm_bytes_per_call")


# ----------------------------------------------------------------- main

PER_CONFIG = ("gqa7b_bf16", "grpo_bf16", "straggler_bf16")   # the other long-tailed GQA decode steps


def time_decode(args, w, dev, shared_prefix=False, op="decode"):
    """Generate one step of workload ``w`` on ``dev`` and time ``args.steps``
    calls after ``args.warmup`` untimed ones. Returns the inputs and the
    measured figures (wall and HIP-event times, single-call spread, status)."""
    import torch

    from paper_2605_20863_amd import _lib
    from paper_2605_20863_amd import workloads as W

    print(f"[bench] generating {w.name}", file=sys.stderr, flush=True)
    inp = W.generate(w, dev)
    lens = inp.layout.seq_lens
    gp = W.group_prefix(w, inp.layout)
    if shared_prefix and gp is None:
        print(f"--shared-prefix needs a GRPO workload (groups sharing prompt blocks); {w.name} has none",
              file=sys.stderr)
        sys.exit(2)
    shared = gp if shared_prefix else None
    nbytes, tokens = algorithmic_bytes(w, lens, shared)
    kv_bytes = inp.k_cache.numel() * inp.k_cache.element_size() * 2
    # rotate over >= 4 GB of cache copies (16x the last-level cache) between steps
    ncopies = max(1, min(16, math.ceil(16 * LLC_BYTES / kv_bytes)))
    caches = [(inp.k_cache, inp.v_cache, inp.kv_scales)]
    for _ in range(ncopies - 1):
        caches.append((inp.k_cache.clone(), inp.v_cache.clone(),
                       inp.kv_scales.clone() if inp.kv_scales is not None else None))
    out = torch.empty_like(inp.q)

    stream = torch.cuda.current_stream(dev)
    prob = _lib.problem_for(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                            inp.layout.max_seq_len, out)
    opts = _lib.make_options(args.variant, args.waves_per_cu, args.min_blocks_per_wave, args.chunks_per_wave,
                             args.min_blocks_per_chunk)
    ptrs = [(k.data_ptr(), v.data_ptr(), s.data_ptr() if s is not None else None) for k, v, s in caches]
    sh = stream.cuda_stream
    qp, bp, lp, op_ = inp.q.data_ptr(), inp.block_table.data_ptr(), inp.seq_lens.data_ptr(), out.data_ptr()

    if shared is not None:
        sb_dev = torch.as_tensor(shared[1], device=dev)

    if op == "append":
        # one new token per sequence, written into its last slot (the block exists)
        gen = torch.Generator(device=dev).manual_seed(7)
        B, hkv, d = len(lens), w.num_kv_heads, w.head_dim
        k_new = torch.randn((B, hkv, d), generator=gen, device=dev).to(torch.bfloat16)
        v_new = torch.randn((B, hkv, d), generator=gen, device=dev).to(torch.bfloat16)
        positions = torch.clamp(inp.seq_lens - 1, min=-1).to(torch.int32)
        aprob = _lib.AppendProblem(B, hkv, d, w.block_size, inp.block_table.shape[1], inp.k_cache.shape[0],
                                   _lib.BF16, _lib._dtype_code(inp.k_cache, "k_cache"))
        nbytes, tokens = append_bytes(w, B), B

    def step(i, sh=sh):
        kp, vp, sp = ptrs[i % ncopies]
        if op == "append":
            rc = _lib.raw_kv_append(k_new.data_ptr(), v_new.data_ptr(), kp, vp, sp, bp, positions.data_ptr(),
                                    aprob, sh)
        elif shared is not None:
            rc = _lib.raw_call_shared_prefix(qp, kp, vp, bp, lp, sp, op_, inp.softmax_scale, shared[0],
                                             sb_dev.data_ptr(), prob, opts, sh)
        else:
            rc = _lib.raw_call(qp, kp, vp, bp, lp, sp, op_, inp.softmax_scale, prob, opts, sh)
        if rc != 0:
            raise RuntimeError(f"pda error {rc}: {_lib.last_error()}")

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    if op == "decode":
        assert torch.isfinite(out.float()).all(), "non-finite output"

    # Timed region: K back-to-back calls. Two HIP events on the calls' stream
    # bracket it (events between calls would add their own GPU time), so the
    # per-call GPU time is the region's event time / K, directly comparable
    # with rocprofv3's decode + combine kernel durations.
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    call_ms = ev0.elapsed_time(ev1) / args.steps
    ms_per_step = wall * 1e3 / args.steps
    spread = per_call_spread(step, args.steps, stream, args.steps)
    status = _lib.read_device_status()
    print(f"[bench] {w.name}: {ms_per_step * 1e3:.1f} us/step wall, {call_ms * 1e3:.1f} us/call GPU "
          f"(HIP events over the timed region), {ncopies} cache copies, status {status}; single calls: "
          f"median {spread['median']} us, min {spread['min']}, max {spread['max']}",
          file=sys.stderr, flush=True)
    traffic = (measured_traffic(w.name + ("_shared" if shared is not None else ""), nbytes)
               if op == "decode" else None)
    graph_ms = graph_call_ms(step, ncopies, args.steps, dev) if op == "decode" and not args.no_graph else None
    del caches, ptrs
    return dict(inp=inp, nbytes=nbytes, tokens=tokens, ncopies=ncopies, call_ms=call_ms, ms_per_step=ms_per_step,
                spread=spread, status=status, traffic=traffic, shared=shared, graph_ms=graph_ms)


def graph_call_ms(step, ncopies, steps, dev):
    """Per-call GPU time of the same calls replayed from a HIP graph: one
    graph holds one call per cache copy (so replays still rotate the copies),
    and it is replayed until at least ``steps`` calls have run, between two
    HIP events on the replay stream. Launch costs of the host drop out; what
    remains is the device's own time per call, gaps between kernels included."""
    import torch

    s = torch.cuda.Stream(dev)
    step(0, s.cuda_stream)  # an eager call sizes the stream's workspace before the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for i in range(ncopies):
            step(i, s.cuda_stream)
    reps = max(1, math.ceil(steps / ncopies))
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(s):
        g.replay()  # warm-up replay
        ev0.record(s)
        for _ in range(reps):
            g.replay()
        ev1.record(s)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / (reps * ncopies)
    del g
    return ms


def graph_fields(nbytes, graph_ms):
    """Per-call figures of the HIP-graph replay (None when not measured)."""
    if graph_ms is None:
        return None
    achieved = nbytes / (graph_ms * 1e-3) / 1e9
    return {"call_us": round(graph_ms * 1e3, 2), "achieved": round(achieved, 2),
            "frac": round(achieved / HBM_PEAK_GBS, 4)}


def per_config_line(args, dev):
    """The other long-tailed GQA decode steps, each generated, timed as the
    headline step is, and freed in turn: per-call GPU time, fraction of peak
    and measured-over-algorithmic HBM bytes."""
    import torch

    from paper_2605_20863_amd import workloads as W

    res = {}
    for name in PER_CONFIG:
        w = W.WORKLOADS[name]
        r = time_decode(args, w, dev)
        achieved = r["nbytes"] / (r["call_ms"] * 1e-3) / 1e9
        res[name] = {
            "call_us": round(r["call_ms"] * 1e3, 2),
            "ms_per_step": round(r["ms_per_step"], 5),
            "achieved": round(achieved, 2),
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "value_wall_gbs": round(r["nbytes"] / (r["ms_per_step"] * 1e-3) / 1e9, 2),
            "algorithmic_bytes_per_call": r["nbytes"],
            "traffic_over_algorithmic": round(r["traffic"] / r["nbytes"], 4) if r["traffic"] else None,
            "kv_tokens_per_s": round(r["tokens"] / (r["call_ms"] * 1e-3), 1),
            "single_call_us": r["spread"],
            "graph_replay": graph_fields(r["nbytes"], r["graph_ms"]),
            "status": r["status"],
        }
        del r
        torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=None,
                    help="default: fp8kv (decode; the largest single-GPU step), gqa7b_bf16 (append), "
                         "logprob_gqa7b_bf16 (prefill)")
    ap.add_argument("--variant", default="auto", choices=["auto", "vector", "mfma"])
    ap.add_argument("--waves-per-cu", type=int, default=0)
    ap.add_argument("--min-blocks-per-wave", type=int, default=0)
    ap.add_argument("--chunks-per-wave", type=int, default=0, help="1 = static split; 0 = library default")
    ap.add_argument("--min-blocks-per-chunk", type=int, default=0)
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle wall time")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="run only a plain 1 GiB device copy (for scaling rocprofv3 byte counters)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="decode: skip the HIP-graph replay timing (profiled runs trace the eager calls only)")
    ap.add_argument("--no-per-config", action="store_true",
                    help="decode: skip timing the other long-tailed GQA steps (" + ", ".join(PER_CONFIG) + ")")
    ap.add_argument("--op", default="decode", choices=["decode", "append", "prefill"],
                    help="decode: one attention step (default); append: the KV append of one decode step "
                         "(each sequence's new token written into its last slot); prefill: the causal varlen "
                         "prefill of a log-prob forward")
    ap.add_argument("--shared-prefix", action="store_true",
                    help="GRPO workloads: read each group's shared prompt blocks once for several members "
                         "(pda_paged_decode_attention_shared_prefix); bytes count the shared blocks once")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (the step shards by sequence "
              "or by KV head with no exchange, but nothing here launches on several GPUs); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2605_20863_amd import workloads as W

    dev = torch.device("cuda:0")
    if args.calibrate_copy:
        # a copy kernel of known size: reads and writes 2^30 bytes per dispatch
        src = torch.randn(1 << 28, device=dev)
        dst = torch.empty_like(src)
        for _ in range(args.warmup + args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "copy", "bytes_read_per_dispatch": 1 << 30,
                          "bytes_written_per_dispatch": 1 << 30, "dispatches": args.warmup + args.steps}))
        return

    if args.workload is None:
        args.workload = {"prefill": "logprob_gqa7b_bf16", "append": "gqa7b_bf16"}.get(args.op, "fp8kv")
    w = W.WORKLOADS[args.workload]
    if (args.op == "prefill") != w.is_prefill:
        print(f"--op {args.op} does not fit workload {w.name}", file=sys.stderr)
        sys.exit(2)
    if args.op == "prefill":
        prefill_main(args, w, dev)
        return
    r = time_decode(args, w, dev, args.shared_prefix, args.op)
    inp, nbytes, tokens, shared = r["inp"], r["nbytes"], r["tokens"], r["shared"]
    call_ms, ms_per_step, traffic = r["call_ms"], r["ms_per_step"], r["traffic"]
    lens = inp.layout.seq_lens

    achieved = nbytes / (call_ms * 1e-3) / 1e9
    value = nbytes / (ms_per_step * 1e-3) / 1e9
    res = {
        "metric": ("paged decode attention achieved HBM GB/s (% of peak) + KV tokens/s read" if args.op == "decode"
                   else "paged KV append achieved HBM GB/s (% of peak) + new tokens/s written"),
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # arithmetic of the path: bf16 products (fp8 codes convert exactly to
        # bf16) with fp32 sums, or fp32 throughout for an fp32 cache
        "dtype": "f32" if w.kv_dtype == "f32" else "bf16",
        "data": "synthetic",
        "pct_of_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "kv_tokens_per_s": round(tokens / (ms_per_step * 1e-3), 1),
        "kv_token_heads_per_s": round(tokens * w.num_kv_heads / (ms_per_step * 1e-3), 1),
        "config": {
            "workload": w.name,
            "num_seqs": len(lens),
            "q_heads": w.num_q_heads,
            "kv_heads": w.num_kv_heads,
            "head_dim": w.head_dim,
            "q_dtype": w.q_dtype,
            "kv_dtype": w.kv_dtype,
            "block_size": w.block_size,
            "total_tokens": tokens,
            "max_seq_len": int(lens.max()),
            "variant": args.variant,
            "cache_copies": r["ncopies"],
            "shared_prefix": shared is not None,
            "q_tokens": w.q_tokens,
            "op": args.op,
        },
        "roofline": {
            "bound": "hbm",
            "kernel": ("KV append (one call)" if args.op == "append"
                       else "decode step (prefix check + stream-K decode + LSE combine, one call)" if shared is not None
                       else "decode step (stream-K decode + LSE combine, one call)"),
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "traffic_over_algorithmic": round(traffic / nbytes, 4) if traffic else None,
            "algorithmic_bytes_per_call": nbytes,
            "call_us": round(call_ms * 1e3, 2),
            "single_call_us": r["spread"],
            "graph_replay": graph_fields(nbytes, r["graph_ms"]),
        },
        "cpu_baseline": None,
    }
    del r
    if not args.no_cpu_baseline and args.op == "decode" and w.q_tokens == 1:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(inp, args.cpu_budget)
        _stop_semaphore_tracker()
    if (args.op == "decode" and not args.shared_prefix and not args.no_per_config
            and args.workload not in PER_CONFIG):
        # the headline step's inputs are freed first: each step is timed on
        # fresh allocations, as it would be in a run of its own
        del inp
        torch.cuda.empty_cache()
        res["per_config"] = per_config_line(args, dev)
    print(json.dumps(res), flush=True)


def prefill_main(args, w, dev):
    """--op prefill: one call = the plan kernel + the attention kernel over all
    packed query tokens of the log-prob forward."""
    import numpy as np
    import torch

    from paper_2605_20863_amd import _lib
    from paper_2605_20863_amd import workloads as W

    print(f"[bench] generating {w.name}", file=sys.stderr, flush=True)
    pin = W.generate_prefill(w, dev)
    c = pin.cache
    lens = c.layout.seq_lens
    flops, pairs = prefill_flops(w, lens, pin.counts)
    T = int(pin.q.shape[0])
    # two cache copies, alternated: a step never starts on the previous step's cached tiles
    caches = [(c.k_cache, c.v_cache, c.kv_scales),
              (c.k_cache.clone(), c.v_cache.clone(), c.kv_scales.clone() if c.kv_scales is not None else None)]
    out = torch.empty_like(pin.q)
    stream = torch.cuda.current_stream(dev)
    prob = _lib.PrefillProblem(len(lens), T, w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size,
                               c.block_table.shape[1], c.k_cache.shape[0], c.layout.max_seq_len, _lib.BF16,
                               _lib._dtype_code(c.k_cache, "k_cache"), _lib.BF16)
    ptrs = [(k.data_ptr(), v.data_ptr(), s.data_ptr() if s is not None else None) for k, v, s in caches]
    sh = stream.cuda_stream
    args_fixed = (pin.q.data_ptr(), pin.q_offsets.data_ptr())

    def step(i):
        kp, vp, sp = ptrs[i % 2]
        rc = _lib.raw_prefill(args_fixed[0], args_fixed[1], kp, vp, c.block_table.data_ptr(), c.seq_lens.data_ptr(),
                              sp, out.data_ptr(), c.softmax_scale, prob, sh)
        if rc != 0:
            raise RuntimeError(f"pda error {rc}: {_lib.last_error()}")

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all(), "non-finite output"
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for i in range(args.steps):
        step(i)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    call_ms = ev0.elapsed_time(ev1) / args.steps
    ms_per_step = wall * 1e3 / args.steps
    spread = per_call_spread(step, args.steps, stream, args.steps)
    status = _lib.read_device_status()
    print(f"[bench] {w.name}: {ms_per_step * 1e3:.1f} us/step wall, {call_ms * 1e3:.1f} us/call GPU, status {status}; "
          f"single calls: median {spread['median']} us, min {spread['min']}, max {spread['max']}",
          file=sys.stderr, flush=True)
    achieved = flops / (call_ms * 1e-3) / 1e12
    value = flops / (ms_per_step * 1e-3) / 1e12
    dtype = {"bf16": "bf16", "fp8_e4m3": "fp8e4m3-kv/bf16-q"}[w.kv_dtype]
    res = {
        "metric": "paged varlen causal prefill achieved TFLOP/s (% of bf16 dense MFMA peak) + query tokens/s",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "pct_of_peak": round(100 * value / MFMA_BF16_PEAK_TFS, 2),
        "tokens_per_s": round(T / (ms_per_step * 1e-3), 1),
        "config": {
            "workload": w.name,
            "num_seqs": len(lens),
            "q_heads": w.num_q_heads,
            "kv_heads": w.num_kv_heads,
            "head_dim": w.head_dim,
            "kv_dtype": w.kv_dtype,
            "block_size": w.block_size,
            "query_tokens": T,
            "cached_tokens": int(lens.sum()),
            "max_seq_len": int(lens.max()),
            "visible_pairs": pairs,
            "op": "prefill",
        },
        "roofline": {
            "bound": "mfma",
            "kernel": "prefill (plan + attention kernel, one call)",
            "achieved": round(achieved, 2),
            "peak": MFMA_BF16_PEAK_TFS,
            "unit": "TFLOP/s",
            "frac": round(achieved / MFMA_BF16_PEAK_TFS, 4),
            "traffic": measured_traffic(w.name, flops, PREFILL_SOURCE),
            "algorithmic_flops_per_call": flops,
            "call_us": round(call_ms * 1e3, 2),
            "single_call_us": spread,
        },
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline_prefill(pin, args.cpu_budget)
        _stop_semaphore_tracker()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
