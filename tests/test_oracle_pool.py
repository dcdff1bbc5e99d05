"""The pooled oracle that the full-size GPU parity tests use (one sequence per
worker job, each job a copy of that sequence's own blocks) gives exactly the
one-process oracle's output, for plain, GRPO (shared blocks), fp8 and
multi-token inputs, including empty sequences; and the prefill's row-slice
jobs (a sequence's query rows split into slices, each a cut of the sequence)
give exactly the one-process prefill oracle. Runs on the CPU."""

import numpy as np
import torch

from paper_2605_20863_amd import workloads as W
from tests import _gpu_util as U
from tests import _oracle_pool as P


def test_pooled_oracle_equals_one_process_oracle():
    for name in ("gqa7b_bf16", "grpo_bf16", "fp8kv", "tiny_mha_f32"):
        w = W.SMALL_WORKLOADS[name]
        inp = W.generate(w, "cpu")
        whole = U.oracle_whole(inp, name)
        assert np.array_equal(whole, U.oracle_for(inp)), name
    lens = [0, 1, 17, 300, 0, 45]
    w = W.Workload("pool_mt", len(lens), 8, 2, 64, "bf16", "fp8_e4m3", ("uniform", 1, 1), cfg_id=55, q_tokens=3)
    inp = W.generate(w, "cpu", seq_lens=lens)
    whole = U.oracle_whole(inp, "multi-token")
    import oracle
    ref = oracle.paged_multi_token_attention(
        q=U.raw(inp.q), k_cache=U.raw(inp.k_cache), v_cache=U.raw(inp.v_cache),
        block_table=inp.layout.block_table, seq_lens=inp.layout.seq_lens, softmax_scale=inp.softmax_scale,
        q_dtype="bf16", kv_dtype="fp8_e4m3", kv_scales=U.raw(inp.kv_scales))
    assert np.array_equal(whole, ref)
    assert P.cores_used() == min(P.cores_available(), P.MAX_CORES)


def test_pooled_prefill_oracle_equals_one_process_oracle():
    import oracle
    for kv in ("bf16", "fp8_e4m3"):
        w = W.Workload(f"pool_pf_{kv}", 5, 8, 2, 64, "bf16", kv, ("uniform", 1, 1), cfg_id=56, prefill_chunk=100)
        # lengths with an empty sequence, one shorter than its chunk and one of
        # several slices; counts include one with tokens at negative positions
        pin = W.generate_prefill(w, "cpu", seq_lens=[0, 40, 300, 17, 129], q_counts=[0, 40, 150, 30, 129])
        c = pin.cache
        ref = oracle.paged_prefill_attention(
            q=U.raw(pin.q), q_offsets=pin.offsets, k_cache=U.raw(c.k_cache), v_cache=U.raw(c.v_cache),
            block_table=c.layout.block_table, seq_lens=c.layout.seq_lens, softmax_scale=c.softmax_scale,
            q_dtype="bf16", kv_dtype=kv, kv_scales=U.raw(c.kv_scales) if c.kv_scales is not None else None)
        whole = U.oracle_prefill_whole(pin, kv, rows_per_job=37)
        assert np.array_equal(whole, ref), kv


def test_worst_row_diagnostic():
    ref = np.ones((2, 3, 4))
    got = ref.copy()
    got[1, 2, 0] += 0.5
    worst, at = U.worst_row_rel_l2(got, ref)
    assert at == (1, 2) and abs(worst - 0.25) < 1e-15
    assert torch.isfinite(torch.tensor(worst))
