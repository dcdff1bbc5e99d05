"""GPU parity: the HIP library (through its C interface) against the fp64 oracle.

Tolerances: max-abs <= 1e-2 and relative L2 <= 5e-3 for bf16 and fp8 caches,
max-abs <= 1e-5 for fp32 -- fp32 accumulation in every kernel, one rounding
of the output to q's dtype.
"""

import time

import numpy as np
import pytest
import torch

import oracle

from paper_2605_20863_amd import workloads as W
from tests import _gpu_util as U

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    from paper_2605_20863_amd import _lib
    return _lib


def run(lib, inp, **opts):
    out = torch.empty_like(inp.q)
    lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                               inp.kv_scales, out, inp.softmax_scale,
                               max_seq_len=inp.layout.max_seq_len, **opts)
    torch.cuda.synchronize()
    return out


def variants_for(w):
    vs = ["auto"]
    if w.group <= 8:
        vs.append("vector")
    if w.kv_dtype != "f32":
        vs.append("mfma")
    return vs


SMALL = sorted(W.SMALL_WORKLOADS)


@pytest.mark.parametrize("name", SMALL)
def test_small_workloads_all_variants(lib, name):
    w = W.SMALL_WORKLOADS[name]
    inp = W.generate(w, DEV)
    ref = U.oracle_for(inp)
    for v in variants_for(w):
        print(f"[parity] {w.name} variant={v}", flush=True)
        got = U.out_to_f64(run(lib, inp, variant=v))
        U.assert_close(got, ref, w.kv_dtype, f"{w.name}/{v}")
    assert lib.read_device_status() == 0


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3", "f32"])
@pytest.mark.parametrize("G", [1, 4, 7, 8])
@pytest.mark.parametrize("D", [64, 128])
def test_edge_lengths(lib, kv, G, D):
    lens = [1, 15, 16, 17, 31, 32, 33, 0, 511, 512, 513, 100]
    w = W.Workload(f"edge_{kv}_{G}_{D}", len(lens), 2 * G, 2, D, "f32" if kv == "f32" else "bf16", kv,
                   ("uniform", 1, 1), cfg_id=90 + G)
    inp = W.generate(w, DEV, seq_lens=lens)
    ref = U.oracle_for(inp)
    vs = variants_for(w)
    for v in vs:
        for split in ({}, {"min_blocks_per_wave": 1, "waves_per_cu": 32}, {"min_blocks_per_wave": 1 << 20},
                      {"chunks_per_wave": 1, "min_blocks_per_wave": 1}):
            print(f"[parity] edge kv={kv} G={G} D={D} variant={v} split={split}", flush=True)
            got = U.out_to_f64(run(lib, inp, variant=v, **split))
            U.assert_close(got, ref, kv, f"edge {kv} G={G} D={D} {v} {split}")
            assert np.array_equal(got[7], np.zeros_like(got[7])), "empty sequence must give zeros"


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("scale", [-0.15, 0.0, 1e-4, 0.3])
def test_softmax_scales(lib, kv, scale):
    """Any finite softmax scale, on both kernel families: a negative scale,
    zero (the mean of the values) and a tiny one."""
    lens = [1, 17, 40, 300, 0, 129]
    w = W.Workload(f"scale_{kv}", len(lens), 8, 2, 128, "bf16", kv, ("uniform", 1, 1), cfg_id=97)
    inp = W.generate(w, DEV, seq_lens=lens)
    ref = oracle.paged_decode_attention(
        q=U.raw(inp.q), k_cache=U.raw(inp.k_cache), v_cache=U.raw(inp.v_cache), block_table=inp.layout.block_table,
        seq_lens=inp.layout.seq_lens, softmax_scale=scale, q_dtype="bf16", kv_dtype=kv,
        kv_scales=U.raw(inp.kv_scales) if inp.kv_scales is not None else None)
    for v in ("vector", "mfma"):
        out = torch.empty(inp.q.shape, dtype=torch.float32, device=DEV)
        lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, inp.kv_scales,
                                   out, scale, variant=v, min_blocks_per_wave=1, waves_per_cu=16)
        torch.cuda.synchronize()
        U.assert_close(U.out_to_f64(out), ref, kv, f"scale {scale} {kv} {v}")
    assert lib.read_device_status() == 0


@pytest.mark.parametrize("name", ["gqa7b_bf16", "fp8kv", "tiny_mha_f32"])
def test_peaked_softmax(lib, name):
    # q x 8 makes logits ~N(0, 64): a few tokens dominate and the running max
    # moves late, stressing the online rescaling and the P rounding. With an
    # fp32 output the kernel's own error is held to the strict bounds; a bf16
    # output may also carry its final rounding (|out| here reaches ~4).
    w = W.SMALL_WORKLOADS[name]
    inp = W.generate(w, DEV, q_scale=8.0)
    ref = U.oracle_for(inp)
    for v in variants_for(w):
        print(f"[parity] peaked {w.name} variant={v}", flush=True)
        out32 = torch.empty(inp.q.shape, dtype=torch.float32, device=DEV)
        lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                                   inp.kv_scales, out32, inp.softmax_scale, variant=v)
        torch.cuda.synchronize()
        U.assert_close(U.out_to_f64(out32), ref, w.kv_dtype, f"peaked {name}/{v} f32 out")
        U.assert_close(U.out_to_f64(run(lib, inp, variant=v)), ref, w.kv_dtype, f"peaked {name}/{v}",
                       bf16_out_rounding=w.q_dtype == "bf16")


# Dynamic split: waves_per_cu = 1 (256 waves) and chunks of 1-3 block-heads, so
# there are several chunks per wave, handed out by the counter, and long
# sequences are cut into hundreds of partials that the combine merges.
# Batches above 512 sequences take the planner's multi-tile path (chunk starts
# found by re-reading seq_lens instead of the LDS copy).
SPLITS = {
    "auto": {},
    "static": {"chunks_per_wave": 1, "min_blocks_per_wave": 1, "waves_per_cu": 1},
    "dynamic": {"chunks_per_wave": 16, "min_blocks_per_chunk": 1, "min_blocks_per_wave": 1, "waves_per_cu": 1},
    "dynamic3": {"chunks_per_wave": 4, "min_blocks_per_chunk": 3, "min_blocks_per_wave": 1, "waves_per_cu": 2},
}


@pytest.mark.parametrize("B", [300, 700, 1100])
@pytest.mark.parametrize("kv,G", [("bf16", 4), ("fp8_e4m3", 8), ("bf16", 2)])
def test_dynamic_split_and_large_batches(lib, B, kv, G):
    rng = np.random.default_rng(B + G)
    lens = np.minimum(np.round(rng.lognormal(np.log(120), 1.0, B)), 4000).astype(int)
    lens[rng.choice(B, B // 20, replace=False)] = 0          # a few empty sequences
    lens[rng.choice(B, 2, replace=False)] = [2500, 3999]   # and two long ones
    w = W.Workload(f"dyn_{kv}_{G}_{B}", B, 2 * G, 2, 64, "bf16", kv, ("uniform", 1, 1), cfg_id=70 + G)
    inp = W.generate(w, DEV, seq_lens=lens.tolist())
    ref = U.oracle_for(inp)
    for v in variants_for(w):
        for name, split in SPLITS.items():
            print(f"[parity] dynamic B={B} kv={kv} G={G} variant={v} split={name}", flush=True)
            got = run(lib, inp, variant=v, **split)
            U.assert_close(U.out_to_f64(got), ref, kv, f"B={B} {kv} G={G} {v} {name}")
            if name.startswith("dynamic"):
                again = run(lib, inp, variant=v, **split)
                assert torch.equal(got.view(torch.int16), again.view(torch.int16)), \
                    "a dynamic split must not change the result"
    assert lib.read_device_status() == 0


def test_deterministic_and_stream(lib):
    w = W.SMALL_WORKLOADS["straggler_bf16"]
    inp = W.generate(w, DEV)
    a = run(lib, inp)
    s = torch.cuda.Stream()
    out = torch.empty_like(inp.q)
    with torch.cuda.stream(s):
        lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                                   inp.kv_scales, out, inp.softmax_scale)
    s.synchronize()
    assert torch.equal(a.view(torch.int16), out.view(torch.int16)), "results must be bitwise reproducible"


def test_out_of_range_inputs_are_contained(lib):
    lens = [40, 70, 5]
    w = W.Workload("badrange", 3, 8, 2, 128, "bf16", "bf16", ("uniform", 1, 1), cfg_id=80)
    inp = W.generate(w, DEV, seq_lens=lens)
    ref = U.oracle_for(inp)
    # a block-table entry past the cache: that block is skipped and flagged
    bt = inp.block_table.clone()
    bt[1, 2] = inp.k_cache.shape[0] + 7
    out = torch.empty_like(inp.q)
    lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, bt, inp.seq_lens, None, out,
                               inp.softmax_scale)
    st = lib.read_device_status()
    assert st & lib.STATUS_BAD_BLOCK
    got = U.out_to_f64(out)
    assert np.isfinite(got).all()
    U.assert_close(got[[0, 2]], ref[[0, 2]], "bf16", "untouched sequences")
    # a length above max_seq_len is clamped to it and flagged
    out2 = torch.empty_like(inp.q)
    lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, None,
                               out2, inp.softmax_scale, max_seq_len=48)
    st = lib.read_device_status()
    assert st & lib.STATUS_LEN_CLAMPED
    lens48 = inp.layout.seq_lens.copy()
    lens48[1] = 48
    ref48 = oracle.paged_decode_attention(
        q=U.raw(inp.q), k_cache=U.raw(inp.k_cache), v_cache=U.raw(inp.v_cache),
        block_table=inp.layout.block_table, seq_lens=lens48, softmax_scale=inp.softmax_scale,
        q_dtype="bf16", kv_dtype="bf16")
    U.assert_close(U.out_to_f64(out2), ref48, "bf16", "clamped length")
    assert lib.read_device_status() == 0


FULL = ["gqa7b_bf16", "grpo_bf16", "straggler_bf16", "fp8kv", "fp8kv_tp8", "qwen30b_bf16", "qwen235b_bf16"]


@pytest.mark.parametrize("name", FULL)
def test_full_size_whole_tensor(lib, name):
    """Full-size workloads in the launch configuration the benchmark times:
    every output (all B x Hq x D) against the oracle, whose sequences run in a
    pool of worker processes. Whole-tensor max-abs and relative L2; the worst
    single row (one sequence and head) is reported beside them."""
    w = W.WORKLOADS[name]
    t0 = time.perf_counter()
    print(f"[parity] full {name}: generating", flush=True)
    inp = W.generate(w, DEV)
    got = U.out_to_f64(run(lib, inp))
    assert lib.read_device_status() == 0
    ref = U.oracle_whole(inp, f"full {name}")
    max_abs, rel_l2 = U.assert_close(got, ref, w.kv_dtype, f"full {name}")
    worst, at = U.worst_row_rel_l2(got, ref)
    print(f"[parity] full {name}: all {got.size} outputs {tuple(got.shape)}: max_abs {max_abs:.2e} "
          f"rel_l2 {rel_l2:.2e}, worst row rel_l2 {worst:.2e} at {tuple(int(i) for i in at)}; "
          f"{time.perf_counter() - t0:.1f} s", flush=True)
    del inp
    torch.cuda.empty_cache()


def test_repeated_calls_and_workspace_reuse(lib):
    """Consecutive calls on one stream reuse one workspace while the number of
    (sequence, KV head) units and partial slots changes between calls; results
    stay correct and bitwise reproducible."""
    small = W.generate(W.SMALL_WORKLOADS["straggler_bf16"], DEV)   # 2 seqs x 8 KV heads
    big = W.generate(W.SMALL_WORKLOADS["fp8kv"], DEV)              # 6 seqs x 8 KV heads
    ref_small, ref_big = U.oracle_for(small), U.oracle_for(big)
    first = None
    for it in range(3):
        for inp, ref, kv in ((small, ref_small, "bf16"), (big, ref_big, "fp8_e4m3")):
            # many waves per CU and tiny shares: every unit is split across waves
            got = run(lib, inp, waves_per_cu=16, min_blocks_per_wave=1)
            U.assert_close(U.out_to_f64(got), ref, kv, f"reuse iteration {it}")
            if inp is small:
                if first is None:
                    first = got.clone()
                assert torch.equal(first.view(torch.int16), got.view(torch.int16))
    assert lib.read_device_status() == 0
