"""Seeded random sweeps of the GPU paths against the fp64 oracle: shapes, cache
and output dtypes, GQA groups, lengths (empty, one token, block edges, ragged
tails), query tokens per sequence, kernel families and work splits are drawn
together, so combinations no hand-written case names are exercised too.
Tolerances as in test_parity_gpu."""

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


def draw_lengths(rng, B, hi):
    lens = np.minimum(np.round(rng.lognormal(np.log(hi / 8), 1.0, B)), hi).astype(int)
    special = [0, 1, 15, 16, 17, 31, 32, 33]
    for i in rng.choice(B, min(B, 4), replace=False):
        lens[i] = special[int(rng.integers(len(special)))]
    return lens


SPLITS = [{}, {"waves_per_cu": 1, "min_blocks_per_wave": 1}, {"waves_per_cu": 3},
          {"waves_per_cu": 16, "min_blocks_per_wave": 1},
          {"chunks_per_wave": 4, "min_blocks_per_chunk": 2, "min_blocks_per_wave": 1, "waves_per_cu": 2},
          {"min_blocks_per_wave": 1 << 20}]


@pytest.mark.parametrize("seed", range(16))
def test_random_decode(lib, seed):
    rng = np.random.default_rng(1000 + seed)
    kv = ["f32", "bf16", "fp8_e4m3"][int(rng.integers(3))]
    D = [64, 128][int(rng.integers(2))]
    hkv = int(rng.integers(1, 4))
    G = int(rng.choice([1, 2, 3, 4, 7, 8] if kv == "f32" else [1, 2, 3, 4, 5, 7, 8, 12, 16]))
    if kv == "f32":
        G = min(G, 8)
    Q = 1
    if kv != "f32" and G <= 16 and rng.random() < 0.4:
        Q = int(rng.integers(2, 32 // G + 1))
    variants = ["auto"]
    if Q == 1 and G <= 8:
        variants.append("vector")
    if kv != "f32":
        variants.append("mfma")
    variant = variants[int(rng.integers(len(variants)))]
    split = SPLITS[int(rng.integers(len(SPLITS)))]
    B = int(rng.integers(1, 41))
    lens = draw_lengths(rng, B, 3000)
    q_dtype = "f32" if kv == "f32" else "bf16"
    w = W.Workload(f"rand{seed}", B, G * hkv, hkv, D, q_dtype, kv, ("uniform", 1, 1), cfg_id=200 + seed, q_tokens=Q)
    inp = W.generate(w, DEV, seq_lens=lens.tolist())
    out_f32 = bool(rng.integers(2)) and q_dtype == "bf16"
    print(f"[random decode {seed}] kv={kv} D={D} Hkv={hkv} G={G} Q={Q} B={B} variant={variant} split={split} "
          f"out={'f32' if out_f32 else q_dtype}", flush=True)
    q = inp.q
    out = torch.empty(q.shape, dtype=torch.float32 if out_f32 else q.dtype, device=DEV)
    lib.paged_decode_attention(q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, inp.kv_scales, out,
                               inp.softmax_scale, max_seq_len=inp.layout.max_seq_len, variant=variant, **split)
    torch.cuda.synchronize()
    lay = inp.layout
    scales = U.raw(inp.kv_scales) if inp.kv_scales is not None else None
    if Q == 1:
        ref = oracle.paged_decode_attention(
            q=U.raw(q), k_cache=U.raw(inp.k_cache), v_cache=U.raw(inp.v_cache), block_table=lay.block_table,
            seq_lens=lay.seq_lens, softmax_scale=inp.softmax_scale, q_dtype=q_dtype, kv_dtype=kv, kv_scales=scales)
    else:
        ref = oracle.paged_multi_token_attention(
            q=U.raw(q), k_cache=U.raw(inp.k_cache), v_cache=U.raw(inp.v_cache), block_table=lay.block_table,
            seq_lens=lay.seq_lens, softmax_scale=inp.softmax_scale, q_dtype=q_dtype, kv_dtype=kv, kv_scales=scales)
    got = U.out_to_f64(out)
    U.assert_close(got, ref, kv, f"random decode {seed}", bf16_out_rounding=not out_f32 and q_dtype == "bf16")
    assert np.array_equal(got[lens == 0], np.zeros_like(got[lens == 0])), "empty sequences give zeros"
    assert lib.read_device_status() == 0


@pytest.mark.parametrize("seed", range(10))
def test_random_prefill(lib, seed):
    rng = np.random.default_rng(2000 + seed)
    kv = ["bf16", "fp8_e4m3"][int(rng.integers(2))]
    D = [64, 128][int(rng.integers(2))]
    hkv = int(rng.integers(1, 4))
    G = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 12, 16]))
    B = int(rng.integers(1, 13))
    lens = draw_lengths(rng, B, 900)
    # query tokens per sequence: all of them, a chunk, none, or more than the
    # cache holds (positions below 0 see nothing)
    counts = []
    for L in lens:
        r = rng.random()
        counts.append(int(L) if r < 0.4 else int(rng.integers(0, L + 1)) if r < 0.85 else int(L + rng.integers(1, 4)))
    if sum(counts) == 0:
        counts[0] = max(1, int(lens[0]))
    w = W.Workload(f"randpf{seed}", B, G * hkv, hkv, D, "bf16", kv, ("uniform", 1, 1), cfg_id=220 + seed,
                   prefill_frac=1.0)
    pin = W.generate_prefill(w, DEV, seq_lens=lens.tolist(), q_counts=counts)
    out_f32 = bool(rng.integers(2))
    print(f"[random prefill {seed}] kv={kv} D={D} Hkv={hkv} G={G} B={B} tokens={sum(counts)} "
          f"out={'f32' if out_f32 else 'bf16'}", flush=True)
    c = pin.cache
    out = torch.full(pin.q.shape, float("nan"), dtype=torch.float32 if out_f32 else torch.bfloat16, device=DEV)
    lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, c.v_cache, c.block_table, c.seq_lens,
                                c.kv_scales, out, c.softmax_scale, max_seq_len=c.layout.max_seq_len)
    torch.cuda.synchronize()
    ref = oracle.paged_prefill_attention(
        q=U.raw(pin.q), q_offsets=pin.offsets, k_cache=U.raw(c.k_cache), v_cache=U.raw(c.v_cache),
        block_table=c.layout.block_table, seq_lens=c.layout.seq_lens, softmax_scale=c.softmax_scale,
        q_dtype="bf16", kv_dtype=kv, kv_scales=U.raw(c.kv_scales) if c.kv_scales is not None else None)
    U.assert_close(U.out_to_f64(out), ref, kv, f"random prefill {seed}", bf16_out_rounding=not out_f32)
    assert lib.read_device_status() == 0
