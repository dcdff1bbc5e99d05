"""The C interface on the host: the library loads, exports what include/pda.h
declares, and rejects bad arguments with the documented codes before any HIP
call (these tests run without a GPU)."""

import ctypes
import math
import subprocess

import pytest

from paper_2605_20863_amd import _lib as L


def prob(**kw):
    base = dict(num_seqs=4, num_q_heads=8, num_kv_heads=2, head_dim=128, block_size=16,
                max_blocks_per_seq=32, num_blocks=200, max_seq_len=0, q_dtype=L.BF16, kv_dtype=L.BF16,
                out_dtype=None)
    base.update(kw)
    if base["out_dtype"] is None:
        base["out_dtype"] = base["q_dtype"]
    return L.Problem(**base)


def test_exports_every_declared_symbol():
    declared = L.header_symbols()
    assert set(declared) == {"pda_paged_decode_attention", "pda_query_plan", "pda_read_device_status",
                             "pda_release_workspaces", "pda_last_error", "pda_version",
                             "pda_paged_decode_attention_shared_prefix", "pda_query_plan_shared_prefix",
                             "pda_paged_kv_append", "pda_paged_prefill_attention",
                             "pda_paged_decode_attention_noalloc"}
    for name in declared:
        assert hasattr(L._lib, name), name
    nm = subprocess.run(["nm", "-D", "--defined-only", L.LIB_PATH], capture_output=True, text=True).stdout
    exported = {line.split()[-1] for line in nm.splitlines() if " T " in line}
    assert set(declared) <= exported
    # nothing else with the public prefix leaks out
    assert {s for s in exported if s.startswith("pda_")} == set(declared)


def test_version():
    assert L.version() == 1


def test_struct_layout_matches_header(tmp_path):
    """ctypes mirrors of the structs agree with the C compiler's layout of pda.h."""
    src = tmp_path / "layout.c"
    src.write_text(r"""
#include <stddef.h>
#include <stdio.h>
#include "pda.h"
#define F(T, m) printf(#T "." #m " %zu\n", offsetof(T, m))
int main(void) {
  printf("pda_problem %zu\npda_options %zu\npda_plan_info %zu\npda_append_problem %zu\n",
         sizeof(pda_problem), sizeof(pda_options), sizeof(pda_plan_info), sizeof(pda_append_problem));
  printf("pda_prefill_problem %zu\n", sizeof(pda_prefill_problem));
  F(pda_prefill_problem, num_blocks); F(pda_prefill_problem, max_seq_len); F(pda_prefill_problem, out_dtype);
  F(pda_append_problem, num_blocks); F(pda_append_problem, kv_dtype);
  F(pda_problem, num_blocks); F(pda_problem, max_seq_len); F(pda_problem, out_dtype);
  F(pda_options, min_blocks_per_wave); F(pda_options, chunks_per_wave); F(pda_options, min_blocks_per_chunk);
  F(pda_plan_info, chunks_max); F(pda_plan_info, workspace_bytes);
  return 0;
}
""")
    exe = tmp_path / "layout"
    import os
    inc = os.path.dirname(L.HEADER_PATH)
    subprocess.run(["gcc", "-std=c11", "-D__HIP_PLATFORM_AMD__", "-I", inc, "-I", "/opt/rocm/include",
                    str(src), "-o", str(exe)], check=True)
    got = dict(line.rsplit(" ", 1) for line in subprocess.run([str(exe)], capture_output=True, text=True,
                                                               check=True).stdout.splitlines())
    assert int(got["pda_problem"]) == ctypes.sizeof(L.Problem)
    assert int(got["pda_options"]) == ctypes.sizeof(L.Options)
    assert int(got["pda_plan_info"]) == ctypes.sizeof(L.PlanInfo)
    assert int(got["pda_append_problem"]) == ctypes.sizeof(L.AppendProblem)
    assert int(got["pda_prefill_problem"]) == ctypes.sizeof(L.PrefillProblem)
    for m in ("num_blocks", "max_seq_len", "out_dtype"):
        assert int(got[f"pda_prefill_problem.{m}"]) == getattr(L.PrefillProblem, m).offset, m
    assert int(got["pda_append_problem.num_blocks"]) == L.AppendProblem.num_blocks.offset
    assert int(got["pda_append_problem.kv_dtype"]) == L.AppendProblem.kv_dtype.offset
    assert int(got["pda_problem.num_blocks"]) == L.Problem.num_blocks.offset
    assert int(got["pda_problem.max_seq_len"]) == L.Problem.max_seq_len.offset
    assert int(got["pda_problem.out_dtype"]) == L.Problem.out_dtype.offset
    assert int(got["pda_options.min_blocks_per_wave"]) == L.Options.min_blocks_per_wave.offset
    assert int(got["pda_plan_info.workspace_bytes"]) == L.PlanInfo.workspace_bytes.offset
    assert int(got["pda_options.chunks_per_wave"]) == L.Options.chunks_per_wave.offset
    assert int(got["pda_options.min_blocks_per_chunk"]) == L.Options.min_blocks_per_chunk.offset
    assert int(got["pda_plan_info.chunks_max"]) == L.PlanInfo.chunks_max.offset


BAD = [
    (dict(num_seqs=-1), L.EINVAL),
    (dict(num_q_heads=0), L.EINVAL),
    (dict(num_q_heads=7, num_kv_heads=2), L.EINVAL),
    (dict(num_q_heads=34, num_kv_heads=2), L.EUNSUPPORTED),
    (dict(head_dim=96), L.EUNSUPPORTED),
    (dict(head_dim=256), L.EUNSUPPORTED),
    (dict(block_size=32), L.EUNSUPPORTED),
    (dict(max_blocks_per_seq=0), L.EINVAL),
    (dict(num_blocks=0), L.EINVAL),
    (dict(max_seq_len=-5), L.EINVAL),
    (dict(max_seq_len=32 * 16 + 1), L.EINVAL),
    (dict(q_dtype=7), L.EINVAL),
    (dict(kv_dtype=9), L.EINVAL),
    (dict(q_dtype=L.FP8_E4M3), L.EUNSUPPORTED),
    (dict(q_dtype=L.BF16, kv_dtype=L.F32), L.EUNSUPPORTED),
    (dict(q_dtype=L.F32, kv_dtype=L.BF16), L.EUNSUPPORTED),
    (dict(q_dtype=L.F32, kv_dtype=L.FP8_E4M3), L.EUNSUPPORTED),
    (dict(num_seqs=1 << 20, max_blocks_per_seq=1 << 12), L.EINVAL),
    (dict(out_dtype=L.FP8_E4M3), L.EINVAL),
    (dict(q_dtype=L.F32, kv_dtype=L.F32, out_dtype=L.BF16), L.EINVAL),
]


@pytest.mark.parametrize("kw,code", BAD, ids=[str(k) for k, _ in BAD])
def test_bad_problem_rejected_on_host(kw, code):
    p = prob(**kw)
    # dummy non-null pointers: validation must reject before dereferencing anything
    rc = L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, p)
    assert rc == code, L.last_error()
    assert L.last_error()
    with pytest.raises(L.PdaError):
        L.query_plan(p)


def test_bad_scale_and_options_rejected():
    for s in (math.nan, math.inf, -math.inf):
        assert L.raw_call(16, 16, 16, 16, 16, 16, 16, s, prob()) == L.EINVAL
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(), L.Options(5, 0, 0)) == L.EINVAL
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(), L.Options(0, -1, 0)) == L.EINVAL
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(), L.Options(0, 0, -3)) == L.EINVAL
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(), L.Options(0, 0, 0, -1)) == L.EINVAL
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(), L.Options(0, 0, 0, 65)) == L.EINVAL
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(), L.Options(0, 0, 0, 0, -2)) == L.EINVAL
    # vector kernel: at most 8 query heads per KV head
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(num_q_heads=32, num_kv_heads=2),
                      L.Options(L.VARIANT_VECTOR, 0, 0)) == L.EUNSUPPORTED
    # MFMA kernel: not for f32 caches
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(q_dtype=L.F32, kv_dtype=L.F32),
                      L.Options(L.VARIANT_MFMA, 0, 0)) == L.EUNSUPPORTED


def test_null_pointers_rejected():
    p = prob()
    for i in range(7):
        if i == 5:
            continue  # kv_scales may be NULL for bf16
        ptrs = [16] * 7
        ptrs[i] = None
        assert L.raw_call(*ptrs, 0.1, p) == L.EINVAL, i
    assert L.raw_call(16, 16, 16, 16, 16, None, 16, 0.1, prob(kv_dtype=L.FP8_E4M3)) == L.EINVAL


def test_misaligned_pointers_rejected():
    # q, caches and out move in 16-byte units; the int32 / f32 arrays need 4 bytes
    for i, bad in ((0, 24), (1, 8), (2, 40), (6, 18), (3, 18), (4, 2), (5, 6)):
        ptrs = [64] * 7
        ptrs[i] = bad
        assert L.raw_call(*ptrs, 0.1, prob()) == L.EINVAL, i
        assert "aligned" in L.last_error()
    assert L.raw_call(*([64] * 7), 0.1, prob(num_seqs=0)) == L.OK


def test_empty_batch_is_a_no_op():
    assert L.raw_call(None, None, None, None, None, None, None, 0.1, prob(num_seqs=0)) == L.OK


@pytest.mark.parametrize("kw,code", BAD, ids=[str(k) for k, _ in BAD])
def test_noalloc_entry_point_validates_like_the_decode_call(kw, code):
    """The no-allocation entry point runs the decode call's host checks before
    any HIP call: the same codes for bad problems, pointers and alignment."""
    assert L.raw_call_noalloc(16, 16, 16, 16, 16, 16, 16, 0.1, prob(**kw)) == code, L.last_error()
    for i in (0, 3, 6):
        ptrs = [16] * 7
        ptrs[i] = None
        assert L.raw_call_noalloc(*ptrs, 0.1, prob()) == L.EINVAL
    ptrs = [64] * 7
    ptrs[1] = 8
    assert L.raw_call_noalloc(*ptrs, 0.1, prob()) == L.EINVAL and "aligned" in L.last_error()
    assert L.raw_call_noalloc(None, None, None, None, None, None, None, 0.1, prob(num_seqs=0)) == L.OK
    assert L.NOALLOC_SCRATCH_BYTES == 32 << 20


def test_query_plan_variants_and_workspace():
    # AUTO: MFMA for bf16/fp8 with G >= 4, vector otherwise
    assert L.query_plan(prob(num_q_heads=8, num_kv_heads=2)).variant == L.VARIANT_MFMA
    assert L.query_plan(prob(num_q_heads=4, num_kv_heads=2)).variant == L.VARIANT_VECTOR
    assert L.query_plan(prob(kv_dtype=L.FP8_E4M3, num_q_heads=64, num_kv_heads=8)).variant == L.VARIANT_MFMA
    assert L.query_plan(prob(q_dtype=L.F32, kv_dtype=L.F32, num_q_heads=4, num_kv_heads=4)).variant == L.VARIANT_VECTOR
    info = L.query_plan(prob(num_seqs=64, num_q_heads=28, num_kv_heads=4), num_compute_units=256)
    assert info.group_size == 7 and info.waves == 256 * 8
    # default split: static, one chunk per wave; one partial slot per (unit, chunk) boundary
    assert info.chunks_max == info.waves
    slots = 64 * 4 + info.chunks_max
    # header + cum + (m, l) + acc, each rounded up to 256 bytes
    up = lambda x: (x + 255) // 256 * 256
    assert info.workspace_bytes == up(64) + up(64 * 4) + 2 * up(slots * 7 * 4) + up(slots * 7 * 128 * 4)
    info = L.query_plan(prob(), L.make_options("vector", waves_per_cu=3), num_compute_units=10)
    assert info.waves == 30 and info.variant == L.VARIANT_VECTOR and info.chunks_max == 30
    info = L.query_plan(prob(), L.make_options(waves_per_cu=3, chunks_per_wave=8), num_compute_units=10)
    assert info.chunks_max == 240  # dynamic split: up to 8 chunks per wave
    with pytest.raises(L.PdaError):
        L.query_plan(prob(), L.make_options(chunks_per_wave=64), num_compute_units=1 << 24)


def test_one_hip_runtime_in_process():
    # the binding maps torch's HIP runtime before libpda.so, so both use one runtime
    import os

    import torch  # noqa: F401

    maps = open("/proc/self/maps").read()
    hip = {os.path.realpath(l.split()[-1]) for l in maps.splitlines() if "libamdhip64" in l}
    hsa = {os.path.realpath(l.split()[-1]) for l in maps.splitlines() if "libhsa-runtime64" in l}
    assert len(hip) == 1 and len(hsa) == 1, (hip, hsa)


def test_shared_prefix_argument_checks():
    p = prob(num_seqs=8, num_q_heads=32, num_kv_heads=8)
    call = lambda gs, sb=16, pr=p, opt=None: L.raw_call_shared_prefix(16, 16, 16, 16, 16, 16, 16, 0.1, gs, sb, pr, opt)
    assert call(0) == L.EINVAL              # group_size < 1
    assert call(3) == L.EINVAL              # 8 sequences are not groups of 3
    assert call(4, sb=None) == L.EINVAL     # shared_blocks missing
    assert call(4, opt=L.make_options("vector")) == L.EUNSUPPORTED
    assert call(4, pr=prob(num_seqs=8, q_dtype=L.F32, kv_dtype=L.F32)) == L.EUNSUPPORTED
    # an empty batch is a no-op
    assert call(4, sb=None, pr=prob(num_seqs=0)) == L.OK


def test_shared_prefix_plan_and_workspace():
    # GRPO step: 256 sequences = 32 groups of 8, 32/8 heads (G = 4): a prefix entry holds up to
    # 32 / G = 8 members (32 query columns, two MFMA N-tiles), so each group's shared blocks form
    # one entry ahead of 256 suffix entries.
    p = prob(num_seqs=256, num_q_heads=32, num_kv_heads=8, max_blocks_per_seq=2048)
    info = L.query_plan_shared_prefix(p, 8, L.make_options(waves_per_cu=4), num_compute_units=256)
    assert info.variant == L.VARIANT_MFMA and info.waves == 1024 and info.chunks_max == 1024
    entries = 32 * 1 + 256
    slots = entries * 8 + info.chunks_max
    up = lambda x: (x + 255) // 256 * 256
    gp = 8 * 4
    assert info.workspace_bytes == (up(64) + up(32 * 4) + up(entries * 4) + 2 * up(slots * gp * 4)
                                    + up(slots * gp * 128 * 4))
    # G = 8, groups of 8: 4 members per entry (32 columns), 2 entries per group
    p8 = prob(num_seqs=64, num_q_heads=64, num_kv_heads=8, max_blocks_per_seq=2048)
    info = L.query_plan_shared_prefix(p8, 8, L.make_options(waves_per_cu=4), num_compute_units=256)
    entries = 8 * 2 + 64
    slots = entries * 8 + info.chunks_max
    assert info.workspace_bytes == (up(64) + up(8 * 4) + up(entries * 4) + 2 * up(slots * 32 * 4)
                                    + up(slots * 32 * 128 * 4))
    # G = 4 with a small group: a G < 4 batch also runs on the MFMA kernel in this mode
    assert L.query_plan_shared_prefix(prob(num_seqs=6, num_q_heads=4, num_kv_heads=4), 2).variant == L.VARIANT_MFMA


def aprob(**kw):
    base = dict(num_seqs=4, num_kv_heads=2, head_dim=128, block_size=16, max_blocks_per_seq=8, num_blocks=64,
                new_dtype=L.BF16, kv_dtype=L.FP8_E4M3)
    base.update(kw)
    return L.AppendProblem(**base)


def test_append_argument_checks():
    ok_ptrs = [16] * 7
    call = lambda pr, ptrs=ok_ptrs: L.raw_kv_append(*ptrs, pr)
    assert call(aprob(num_seqs=-1)) == L.EINVAL
    assert call(aprob(num_kv_heads=0)) == L.EINVAL
    assert call(aprob(head_dim=96)) == L.EUNSUPPORTED
    assert call(aprob(block_size=32)) == L.EUNSUPPORTED
    assert call(aprob(max_blocks_per_seq=0)) == L.EINVAL
    assert call(aprob(num_blocks=0)) == L.EINVAL
    assert call(aprob(new_dtype=L.FP8_E4M3)) == L.EINVAL
    assert call(aprob(kv_dtype=7)) == L.EINVAL
    for i in range(7):       # every pointer is required (kv_scales because the cache is fp8)
        ptrs = list(ok_ptrs)
        ptrs[i] = None
        assert call(aprob(), ptrs) == L.EINVAL, i
    assert call(aprob(num_seqs=0), [None] * 7) == L.OK   # empty batch: no-op


def test_append_binding_checks_block_table_rows():
    """The append kernel reads block_table[b, :] for every new token b, so the
    binding refuses a table without exactly B rows (or not 2-D) before it
    looks at devices: a short table would be read past its end."""
    import torch

    B, hkv, d, nb = 3, 2, 64, 10
    k_new = torch.zeros((B, hkv, d), dtype=torch.bfloat16)
    v_new = torch.zeros_like(k_new)
    kc = torch.zeros((nb, hkv, 16, d), dtype=torch.bfloat16)
    vc = torch.zeros((nb, hkv, d, 16), dtype=torch.bfloat16)
    pos = torch.zeros(B, dtype=torch.int32)
    for bad in (torch.zeros((B - 1, 4), dtype=torch.int32), torch.zeros((B + 1, 4), dtype=torch.int32),
                torch.zeros(4 * B, dtype=torch.int32)):
        with pytest.raises(ValueError, match="block_table"):
            L.paged_kv_append(k_new, v_new, kc, vc, None, bad, pos)
    with pytest.raises(ValueError, match="k_new"):
        L.paged_kv_append(k_new[0], v_new[0], kc, vc, None, torch.zeros((B, 4), dtype=torch.int32), pos)
    # right shapes pass the shape checks and stop at the device check
    with pytest.raises(ValueError, match="must be on"):
        L.paged_kv_append(k_new, v_new, kc, vc, None, torch.zeros((B, 4), dtype=torch.int32), pos)


def test_multi_token_checks_and_plan():
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(q_tokens=-1)) == L.EINVAL
    # several query tokens need the MFMA kernel (bf16 / fp8 cache) and Q * G <= 32
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1,
                      prob(q_tokens=2, q_dtype=L.F32, kv_dtype=L.F32)) == L.EUNSUPPORTED
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(q_tokens=9)) == L.EUNSUPPORTED   # G = 4: 36 columns
    assert L.raw_call(16, 16, 16, 16, 16, 16, 16, 0.1, prob(q_tokens=4),
                      L.make_options("vector")) == L.EUNSUPPORTED
    assert L.raw_call_shared_prefix(16, 16, 16, 16, 16, 16, 16, 0.1, 2, 16, prob(q_tokens=2)) == L.EUNSUPPORTED
    # Q = 4, G = 2: MFMA (even though G < 4), partial rows of Q * G = 8 columns
    p = prob(num_seqs=64, num_q_heads=8, num_kv_heads=4, q_tokens=4)
    info = L.query_plan(p, L.make_options(waves_per_cu=4), num_compute_units=256)
    assert info.variant == L.VARIANT_MFMA
    slots = 64 * 4 + info.chunks_max
    up = lambda x: (x + 255) // 256 * 256
    assert info.workspace_bytes == up(64) + up(64 * 4) + 2 * up(slots * 8 * 4) + up(slots * 8 * 128 * 4)
    # Q = 8, G = 4: 32 columns (the two-tile kernel), partial rows of 32 columns
    p = prob(num_seqs=64, num_q_heads=8, num_kv_heads=2, q_tokens=8)
    info = L.query_plan(p, L.make_options(waves_per_cu=4), num_compute_units=256)
    assert info.variant == L.VARIANT_MFMA
    slots = 64 * 2 + info.chunks_max
    assert info.workspace_bytes == up(64) + up(64 * 4) + 2 * up(slots * 32 * 4) + up(slots * 32 * 128 * 4)


def pprob(**kw):
    base = dict(num_seqs=4, num_tokens=100, num_q_heads=8, num_kv_heads=2, head_dim=128, block_size=16,
                max_blocks_per_seq=8, num_blocks=64, max_seq_len=0, q_dtype=L.BF16, kv_dtype=L.BF16,
                out_dtype=L.BF16)
    base.update(kw)
    return L.PrefillProblem(**base)


def test_prefill_argument_checks():
    ok_ptrs = [16] * 8
    call = lambda pr, ptrs=ok_ptrs, scale=0.1: L.raw_prefill(*ptrs[:7], ptrs[7], scale, pr)
    assert call(pprob(num_seqs=-1)) == L.EINVAL
    assert call(pprob(num_tokens=-1)) == L.EINVAL
    assert call(pprob(num_kv_heads=3)) == L.EINVAL              # 8 % 3
    assert call(pprob(num_q_heads=34, num_kv_heads=2)) == L.EUNSUPPORTED   # G = 17
    assert call(pprob(head_dim=96)) == L.EUNSUPPORTED
    assert call(pprob(block_size=32)) == L.EUNSUPPORTED
    assert call(pprob(max_blocks_per_seq=0)) == L.EINVAL
    assert call(pprob(num_blocks=0)) == L.EINVAL
    assert call(pprob(max_seq_len=8 * 16 + 1)) == L.EINVAL
    assert call(pprob(q_dtype=L.F32)) == L.EUNSUPPORTED
    assert call(pprob(q_dtype=L.FP8_E4M3)) == L.EINVAL
    assert call(pprob(kv_dtype=L.F32)) == L.EUNSUPPORTED
    assert call(pprob(kv_dtype=5)) == L.EINVAL
    assert call(pprob(out_dtype=L.FP8_E4M3)) == L.EINVAL
    assert call(pprob(), scale=math.inf) == L.EINVAL
    assert call(pprob(num_tokens=2 ** 30, num_q_heads=8)) == L.EINVAL   # T * Hq overflows int32
    # ~17M one-token tiles x 16 KV heads: more units than 8 * unit + queue can name in an int32
    assert call(pprob(num_seqs=17_000_000, num_tokens=1, num_q_heads=16, num_kv_heads=16)) == L.EINVAL
    assert "work units" in L.last_error()
    for i in range(8):
        ptrs = list(ok_ptrs)
        ptrs[i] = None
        # kv_scales (index 6) is optional for a bf16 cache, required for fp8
        want = L.OK if i == 6 else L.EINVAL
        if want == L.OK:
            assert call(pprob(kv_dtype=L.FP8_E4M3), ptrs) == L.EINVAL
        else:
            assert call(pprob(), ptrs) == L.EINVAL, i
    # q (0), k_cache (2), v_cache (3), out (7) need 16-byte alignment; q_offsets (1), table (4), lens (5) 4
    for i, bad in ((0, 24), (2, 8), (3, 40), (7, 20), (1, 2), (4, 6), (5, 18)):
        ptrs = list(ok_ptrs)
        ptrs[i] = bad
        assert call(pprob(), ptrs) == L.EINVAL, i
        assert "aligned" in L.last_error()
    assert call(pprob(num_seqs=0), [None] * 8) == L.OK      # empty batch: no-op
    assert call(pprob(num_tokens=0), [None] * 8) == L.OK    # no query rows: no-op
