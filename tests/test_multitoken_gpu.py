"""GPU parity of multi-token decode (several new query tokens per sequence,
causal over the cache, as in speculative verification) against the fp64
oracle ``oracle.paged_multi_token_attention``. Tolerances as in
test_parity_gpu."""

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


def queries(inp, Q, seed, scale=1.0):
    g = torch.Generator(device=DEV).manual_seed(seed)
    B, hq, d = inp.q.shape
    return (torch.randn((B, Q, hq, d), generator=g, device=DEV) * scale).to(torch.bfloat16)


def run(lib, inp, q, out_dtype=None, **opts):
    out = torch.empty(q.shape, dtype=out_dtype or q.dtype, device=DEV)
    lib.paged_decode_attention(q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, inp.kv_scales, out,
                               inp.softmax_scale, max_seq_len=inp.layout.max_seq_len, **opts)
    torch.cuda.synchronize()
    return out


def reference(inp, q, seqs=None):
    lay = inp.layout
    if seqs is None:
        return oracle.paged_multi_token_attention(
            q=U.raw(q), k_cache=U.raw(inp.k_cache), v_cache=U.raw(inp.v_cache), block_table=lay.block_table,
            seq_lens=lay.seq_lens, softmax_scale=inp.softmax_scale, q_dtype="bf16", kv_dtype=inp.workload.kv_dtype,
            kv_scales=U.raw(inp.kv_scales) if inp.kv_scales is not None else None)
    return oracle.paged_multi_token_attention(
        q=U.raw(q), k_cache=U.raw(inp.k_cache), v_cache=U.raw(inp.v_cache), block_table=lay.block_table,
        seq_lens=lay.seq_lens, softmax_scale=inp.softmax_scale, q_dtype="bf16", kv_dtype=inp.workload.kv_dtype,
        kv_scales=U.raw(inp.kv_scales) if inp.kv_scales is not None else None, seqs=seqs)


SPLITS = {
    "auto": {},
    "many_partials": {"waves_per_cu": 32, "min_blocks_per_wave": 1},
    "dynamic": {"chunks_per_wave": 16, "min_blocks_per_chunk": 1, "min_blocks_per_wave": 1, "waves_per_cu": 1},
    "unsplit": {"min_blocks_per_wave": 1 << 20},
}

# (Q, Hq, Hkv, D, kv): Q * G columns from 6 to 32 (above 16: the two-tile
# body, whose second tile is partly or wholly used)
CASES = [(2, 8, 2, 128, "bf16"), (4, 16, 4, 128, "bf16"), (3, 8, 4, 64, "bf16"), (8, 16, 8, 64, "bf16"),
         (16, 8, 8, 128, "bf16"), (4, 16, 4, 128, "fp8_e4m3"), (2, 64, 8, 128, "fp8_e4m3"),
         (4, 28, 4, 128, "bf16"), (8, 8, 2, 128, "bf16"), (32, 4, 4, 64, "bf16"), (17, 4, 4, 128, "bf16"),
         (9, 4, 2, 128, "fp8_e4m3"), (3, 56, 8, 64, "fp8_e4m3")]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"Q{c[0]}_G{c[1] // c[2]}_D{c[3]}_{c[4]}")
def test_multitoken_edge_lengths(lib, case):
    Q, hq, hkv, d, kv = case
    lens = [1, 2, 3, 15, 16, 17, 31, 32, 33, 0, 100, 513, 18, 47]
    w = W.Workload(f"mt_{Q}_{hq}_{hkv}_{d}_{kv}", len(lens), hq, hkv, d, "bf16", kv, ("uniform", 1, 1),
                   cfg_id=50 + Q)
    inp = W.generate(w, DEV, seq_lens=lens)
    q = queries(inp, Q, seed=Q * 7 + hq)
    ref = reference(inp, q)
    for name, split in SPLITS.items():
        print(f"[parity] multi-token {w.name} split={name}", flush=True)
        # the kernel's own error: fp32 output at the strict bounds; the bf16
        # output may add its rounding (outputs of 1-3-token sequences are single
        # V rows, up to |4|, where bf16 rounding alone exceeds 1e-2)
        got32 = U.out_to_f64(run(lib, inp, q, out_dtype=torch.float32, **split))
        U.assert_close(got32, ref, kv, f"{w.name} {name} f32 out")
        got = U.out_to_f64(run(lib, inp, q, **split))
        U.assert_close(got, ref, kv, f"{w.name} {name}", bf16_out_rounding=True)
        for g in (got, got32):
            assert not g[9].any(), "empty sequence must give zeros"
            assert not g[0, :Q - 1].any(), "queries with no visible token give zeros"
    assert lib.read_device_status() == 0


def test_multitoken_peaked_fp32_out(lib):
    """q x 8 (a few tokens dominate, the max moves late) with an fp32 output:
    the kernel's own error at the strict bounds."""
    w = W.SMALL_WORKLOADS["gqa7b_bf16"].replace(name="mt_peaked", num_q_heads=8, num_kv_heads=4)
    inp = W.generate(w, DEV)
    q = queries(inp, 4, seed=5, scale=8.0)
    ref = reference(inp, q)
    got = U.out_to_f64(run(lib, inp, q, out_dtype=torch.float32))
    U.assert_close(got, ref, "bf16", "peaked multi-token f32 out")


def test_multitoken_full_size_whole_tensor(lib):
    """Speculative verification of 4 tokens at full size on one N-tile (the
    7B lengths with 8 / 2 heads: G = 4, 16 columns), every output against the
    oracle."""
    w = W.WORKLOADS["gqa7b_bf16"].replace(name="mt_full", num_q_heads=8, num_kv_heads=2)
    inp = W.generate(w, DEV)
    q = queries(inp, 4, seed=9)
    got = run(lib, inp, q)
    got = U.out_to_f64(got)
    ref = U.oracle_whole(inp, "multi-token full size", q=q)
    max_abs, rel_l2 = U.assert_close(got, ref, "bf16", "multi-token full size")
    worst, at = U.worst_row_rel_l2(got, ref)
    print(f"[parity] multi-token full size: all {got.size} outputs: max_abs {max_abs:.2e} rel_l2 {rel_l2:.2e}, "
          f"worst row rel_l2 {worst:.2e} at {tuple(int(i) for i in at)}", flush=True)
    assert lib.read_device_status() == 0


def test_multitoken_wide_full_size_whole_tensor(lib):
    """4 query tokens on the 7B GQA step itself (28 / 4 heads, G = 7: 28
    columns in the two-tile body), every output against the oracle."""
    w = W.WORKLOADS["spec4_gqa7b_bf16"]
    inp = W.generate(w, DEV)
    q = inp.q                                   # [64, 4, 28, 128]
    assert q.shape[1] == 4
    got = run(lib, inp, q)
    got = U.out_to_f64(got)
    ref = U.oracle_whole(inp, "wide multi-token full size", q=q)
    max_abs, rel_l2 = U.assert_close(got, ref, "bf16", "wide multi-token full size")
    worst, at = U.worst_row_rel_l2(got, ref)
    print(f"[parity] wide multi-token full size: all {got.size} outputs: max_abs {max_abs:.2e} rel_l2 {rel_l2:.2e}, "
          f"worst row rel_l2 {worst:.2e} at {tuple(int(i) for i in at)}", flush=True)
    assert lib.read_device_status() == 0


def test_multitoken_wide_fp8_full_size_whole_tensor(lib):
    """4 query tokens on the fp8 step's TP-8 share at full size (8 / 1 heads,
    G = 8: all 32 columns of the two-tile body, fp8 e4m3 cache with per-block
    scales, lengths up to 64k), every output against the oracle."""
    w = W.WORKLOADS["fp8kv_tp8"].replace(name="mt_fp8_wide", q_tokens=4)
    inp = W.generate(w, DEV)
    q = inp.q
    assert q.shape[1] == 4
    got = run(lib, inp, q)
    got = U.out_to_f64(got)
    ref = U.oracle_whole(inp, "wide multi-token fp8 full size", q=q)
    max_abs, rel_l2 = U.assert_close(got, ref, "fp8_e4m3", "wide multi-token fp8 full size")
    worst, at = U.worst_row_rel_l2(got, ref)
    print(f"[parity] wide multi-token fp8 full size: all {got.size} outputs: max_abs {max_abs:.2e} rel_l2 {rel_l2:.2e}, "
          f"worst row rel_l2 {worst:.2e} at {tuple(int(i) for i in at)}", flush=True)
    assert lib.read_device_status() == 0
