"""GPU parity of the varlen paged prefill (pda_paged_prefill_attention) against
the fp64 oracle ``oracle.paged_prefill_attention``: packed query tokens, each
causal over its sequence's cache. Tolerances as in test_parity_gpu (bf16 and
fp8 caches: max-abs 1e-2 and relative L2 5e-3, fp32 accumulation)."""

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


@pytest.fixture(params=["image", "staging"])
def path(request, monkeypatch):
    """The attention kernel's two ways of bringing K and V tiles to LDS: direct
    loads from the converted image (the default whenever the image fits), or
    registers and conversion in the kernel (PDA_PREFILL_IMAGE_MAX_MB = 0, as
    for an image larger than the cap)."""
    if request.param == "staging":
        monkeypatch.setenv("PDA_PREFILL_IMAGE_MAX_MB", "0")
    else:
        monkeypatch.delenv("PDA_PREFILL_IMAGE_MAX_MB", raising=False)
    return request.param


def wl(hq, hkv, d, kv, cfg=40):
    return W.Workload(f"prefill_{hq}_{hkv}_{d}_{kv}", 1, hq, hkv, d, "bf16", kv, ("uniform", 1, 1), cfg_id=cfg,
                      prefill_frac=1.0)


def run(lib, pin, out_dtype=torch.bfloat16, out=None):
    c = pin.cache
    if out is None:
        out = torch.full(pin.q.shape, float("nan"), dtype=out_dtype, device=DEV)
    lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, c.v_cache, c.block_table, c.seq_lens, c.kv_scales,
                                out, c.softmax_scale, max_seq_len=c.layout.max_seq_len)
    torch.cuda.synchronize()
    return out


def reference(pin, seqs=None):
    c = pin.cache
    return oracle.paged_prefill_attention(
        q=U.raw(pin.q), q_offsets=pin.offsets, k_cache=U.raw(c.k_cache), v_cache=U.raw(c.v_cache),
        block_table=c.layout.block_table, seq_lens=c.layout.seq_lens, softmax_scale=c.softmax_scale,
        q_dtype="bf16", kv_dtype=c.workload.kv_dtype,
        kv_scales=U.raw(c.kv_scales) if c.kv_scales is not None else None, seqs=seqs)


def check(lib, pin, what, out_dtype=torch.float32):
    out = run(lib, pin, out_dtype)
    ref = reference(pin)
    got = U.out_to_f64(out)
    res = U.assert_close(got, ref, pin.cache.workload.kv_dtype, what,
                         bf16_out_rounding=out_dtype == torch.bfloat16)
    assert lib.read_device_status() == 0
    return res


# (Hq, Hkv): G = 1, 2, 3 (tiles of 85 tokens, one column unused), 4, 7 (the 7B
# model's group), 8, 16 (tiles of 16 tokens)
GROUPS = [(4, 4), (4, 2), (6, 2), (8, 2), (14, 2), (8, 1), (16, 1)]


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("hq,hkv", GROUPS)
def test_prefill_matches_oracle(lib, path, kv, d, hq, hkv):
    """Full prefills (n = L) of ragged sequences spanning several tiles, and
    chunked prefills (n < L) of the same caches."""
    lens = [1, 15, 16, 17, 33, 100, 257, 700]
    counts = [1, 15, 16, 5, 33, 64, 257, 300]
    print(f"[prefill] kv={kv} D={d} Hq={hq} Hkv={hkv}", flush=True)
    pin = W.generate_prefill(wl(hq, hkv, d, kv), DEV, seq_lens=lens, q_counts=counts)
    check(lib, pin, f"{kv} D{d} G{hq // hkv}")


# (Hq, Hkv, D): the attention grid's unit queues, gcd(Hkv, 8) of them, each
# holding Hkv / gcd(Hkv, 8) KV heads: 8 queues of one head, 8 of two, 2 of
# three, one of five. The lengths give more units than the grid has
# workgroups, so most units are claimed from the counters, and queues drain
# at different times, so workgroups take units from other queues.
QUEUE_SHAPES = [(16, 8, 64), (16, 16, 64), (18, 6, 128), (15, 5, 64)]


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("hq,hkv,d", QUEUE_SHAPES)
def test_prefill_queues_more_units_than_workgroups(lib, kv, hq, hkv, d):
    lens = [1300, 41, 2100, 700, 1650, 5, 999]
    counts = [1300, 41, 1500, 700, 1650, 5, 640]
    pin = W.generate_prefill(wl(hq, hkv, d, kv), DEV, seq_lens=lens, q_counts=counts)
    tq = 256 // (hq // hkv)
    units = sum((n + tq - 1) // tq for n in counts) * hkv
    cus = torch.cuda.get_device_properties(DEV).multi_processor_count
    print(f"[prefill queues] kv={kv} Hq={hq} Hkv={hkv} D={d} units={units} CUs={cus}", flush=True)
    assert units > cus, (units, cus)
    out = run(lib, pin, torch.float32)
    ref = U.oracle_prefill_whole(pin, f"queues Hq{hq} Hkv{hkv}")
    U.assert_close(U.out_to_f64(out), ref, kv, f"queues Hq{hq} Hkv{hkv} {kv}")
    assert lib.read_device_status() == 0


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
@pytest.mark.parametrize("hq,hkv,d", [(28, 4, 128), (8, 2, 64), (16, 1, 128), (15, 5, 64)])
def test_prefill_paths_agree_bitwise(lib, monkeypatch, kv, hq, hkv, d):
    """The image and staging paths convert V (and fp8 K) with the same
    functions and run the same products in the same order: their outputs
    agree bit for bit, and the image path matches the oracle."""
    pin = W.generate_prefill(wl(hq, hkv, d, kv), DEV, seq_lens=[40, 700, 129, 5, 300],
                             q_counts=[40, 700, 2, 5, 17])
    monkeypatch.delenv("PDA_PREFILL_IMAGE_MAX_MB", raising=False)
    img = run(lib, pin, torch.float32)
    monkeypatch.setenv("PDA_PREFILL_IMAGE_MAX_MB", "0")
    stg = run(lib, pin, torch.float32)
    assert torch.equal(img.view(torch.int32), stg.view(torch.int32))
    U.assert_close(U.out_to_f64(img), reference(pin), kv, f"paths Hq{hq} Hkv{hkv} D{d} {kv}")
    assert lib.read_device_status() == 0


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_prefill_bf16_output(lib, kv):
    pin = W.generate_prefill(wl(28, 4, 128, kv), DEV, seq_lens=[40, 300, 129], q_counts=[40, 300, 2])
    check(lib, pin, f"bf16 out {kv}", out_dtype=torch.bfloat16)


def test_prefill_edge_counts(lib, path):
    """Empty sequences, queries beyond the cache (n > L: positions below 0 give
    zeros), an empty cache with queries, single tokens, and a sequence long
    enough for many tiles."""
    lens = [0, 5, 0, 20, 1, 3000, 48]
    counts = [0, 9, 3, 0, 1, 3000, 48]
    pin = W.generate_prefill(wl(16, 2, 128, "bf16"), DEV, seq_lens=lens, q_counts=counts)
    check(lib, pin, "edge counts")
    got = U.out_to_f64(run(lib, pin, torch.float32))
    off = pin.offsets
    assert not got[off[1]:off[1] + 4].any()       # positions -4 .. -1 of sequence 1
    assert not got[off[2]:off[3]].any()           # sequence 2 has no cached token


def test_prefill_many_tiny_sequences(lib, path):
    """More sequences than the plan kernel has threads: 2500 sequences of 0 to
    3 queries each."""
    rng = np.random.default_rng(7)
    lens = rng.integers(0, 40, 2500)
    counts = np.minimum(rng.integers(0, 4, 2500), np.maximum(lens, 0))
    pin = W.generate_prefill(wl(8, 2, 64, "fp8_e4m3"), DEV, seq_lens=lens, q_counts=counts)
    check(lib, pin, "2500 tiny sequences")


def test_prefill_untouched_rows_and_determinism(lib):
    """Rows before q_offsets[0] and after q_offsets[B] are not written, and two
    calls give identical bits."""
    pin = W.generate_prefill(wl(8, 2, 128, "bf16"), DEV, seq_lens=[90, 200], q_counts=[90, 150])
    T = pin.q.shape[0]
    q = torch.cat([torch.zeros((3, 8, 128), dtype=torch.bfloat16, device=DEV), pin.q,
                   torch.zeros((5, 8, 128), dtype=torch.bfloat16, device=DEV)])
    offs = torch.from_numpy(pin.offsets + 3).to(DEV)
    c = pin.cache
    outs = []
    for _ in range(2):
        out = torch.full(q.shape, 7.0, dtype=torch.float32, device=DEV)
        lib.paged_prefill_attention(q, offs, c.k_cache, c.v_cache, c.block_table, c.seq_lens, c.kv_scales, out,
                                    c.softmax_scale)
        torch.cuda.synchronize()
        outs.append(out.cpu())
    assert torch.equal(outs[0], outs[1])
    assert (outs[0][:3] == 7.0).all() and (outs[0][3 + T:] == 7.0).all()
    U.assert_close(outs[0][3:3 + T].double().numpy(), reference(pin), "bf16", "offset rows")


def test_prefill_status_bits(lib, path):
    pin = W.generate_prefill(wl(8, 2, 128, "bf16"), DEV, seq_lens=[40, 70], q_counts=[40, 70])
    c = pin.cache
    out = torch.full(pin.q.shape, 7.0, dtype=torch.float32, device=DEV)
    # decreasing offsets: nothing is written, bit 8
    bad = torch.tensor([0, 70, 40], dtype=torch.int32, device=DEV)
    lib.paged_prefill_attention(pin.q, bad, c.k_cache, c.v_cache, c.block_table, c.seq_lens, c.kv_scales, out,
                                c.softmax_scale)
    assert lib.read_device_status() == lib.STATUS_BAD_OFFSETS
    assert (out.cpu() == 7.0).all()
    # an offset past T: the same
    bad = torch.tensor([0, 40, 111], dtype=torch.int32, device=DEV)
    lib.paged_prefill_attention(pin.q, bad, c.k_cache, c.v_cache, c.block_table, c.seq_lens, c.kv_scales, out,
                                c.softmax_scale)
    assert lib.read_device_status() == lib.STATUS_BAD_OFFSETS
    # a length above max_seq_len is clamped (bit 1); the rest is computed
    lens = torch.tensor([40, 71], dtype=torch.int32, device=DEV)
    lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, c.v_cache, c.block_table, lens, c.kv_scales, out,
                                c.softmax_scale, max_seq_len=70)
    assert lib.read_device_status() == lib.STATUS_LEN_CLAMPED
    U.assert_close(U.out_to_f64(out), reference(pin), "bf16", "clamped length")
    # a block id out of range: skipped, bit 2
    table = c.block_table.clone()
    table[1, 2] = c.k_cache.shape[0] + 5
    lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, c.v_cache, table, c.seq_lens, c.kv_scales, out,
                                c.softmax_scale)
    assert lib.read_device_status() == lib.STATUS_BAD_BLOCK
    U.assert_close(U.out_to_f64(out)[:40], reference(pin)[:40], "bf16", "sequence without bad blocks")


@pytest.mark.parametrize("scale", [-0.2, 0.0, 1e-3, 0.7])
def test_prefill_softmax_scales(lib, scale):
    """Any finite softmax scale: a negative one enters through q's sign, zero
    averages the visible values."""
    pin = W.generate_prefill(wl(8, 2, 64, "fp8_e4m3"), DEV, seq_lens=[3, 70, 200], q_counts=[3, 70, 120])
    c = pin.cache
    out = torch.empty(pin.q.shape, dtype=torch.float32, device=DEV)
    lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, c.v_cache, c.block_table, c.seq_lens, c.kv_scales,
                                out, scale)
    torch.cuda.synchronize()
    ref = oracle.paged_prefill_attention(
        q=U.raw(pin.q), q_offsets=pin.offsets, k_cache=U.raw(c.k_cache), v_cache=U.raw(c.v_cache),
        block_table=c.layout.block_table, seq_lens=c.layout.seq_lens, softmax_scale=scale, q_dtype="bf16",
        kv_dtype="fp8_e4m3", kv_scales=U.raw(c.kv_scales))
    U.assert_close(U.out_to_f64(out), ref, "fp8_e4m3", f"scale {scale}")
    assert lib.read_device_status() == 0


def test_prefill_value_range_flag(lib, path):
    """P . V runs in fp16: a live V value beyond +-65504 saturates and sets
    status bit 16; values in range, and poison in dead slots, do not."""
    pin = W.generate_prefill(wl(8, 2, 128, "bf16"), DEV, seq_lens=[40, 70], q_counts=[40, 70])
    c = pin.cache
    out = torch.empty(pin.q.shape, dtype=torch.float32, device=DEV)
    v = c.v_cache.clone()
    p = int(c.layout.block_table[1, 1])
    v[p, 0, 5, 3] = 60000.0            # in range: no flag (token 19 of sequence 1)
    lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, v, c.block_table, c.seq_lens, None, out,
                                c.softmax_scale)
    assert lib.read_device_status() == 0
    v[p, 0, 5, 3] = 1.0e6
    lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, v, c.block_table, c.seq_lens, None, out,
                                c.softmax_scale)
    assert lib.read_device_status() == lib.STATUS_HALF_RANGE
    assert torch.isfinite(out).all()


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_prefill_shared_blocks(lib, path, kv):
    """Sequences that share their leading physical blocks, as the rollouts of
    one GRPO group share their prompt's: on the image path several workgroups
    convert the same tiles (writing the same bytes). Against the oracle with
    the same shared table."""
    pin = W.generate_prefill(wl(28, 4, 128, kv), DEV, seq_lens=[300, 170, 260, 49, 333, 95],
                             q_counts=[300, 170, 200, 49, 12, 95])
    c = pin.cache
    table = c.layout.block_table.copy()
    shared = 3  # every sequence's first 48 tokens live in sequence 0's first three blocks
    table[1:, :shared] = table[0, :shared]
    tdev = torch.from_numpy(table).to(DEV)
    out = torch.full(pin.q.shape, float("nan"), dtype=torch.float32, device=DEV)
    lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, c.v_cache, tdev, c.seq_lens, c.kv_scales, out,
                                c.softmax_scale, max_seq_len=c.layout.max_seq_len)
    torch.cuda.synchronize()
    ref = oracle.paged_prefill_attention(
        q=U.raw(pin.q), q_offsets=pin.offsets, k_cache=U.raw(c.k_cache), v_cache=U.raw(c.v_cache),
        block_table=table, seq_lens=c.layout.seq_lens, softmax_scale=c.softmax_scale, q_dtype="bf16",
        kv_dtype=kv, kv_scales=U.raw(c.kv_scales) if c.kv_scales is not None else None)
    U.assert_close(U.out_to_f64(out), ref, kv, f"shared blocks {kv} ({path})")
    assert lib.read_device_status() == 0


def test_prefill_after_appends(lib):
    """A cache written token by token by the append kernel, then read by the
    prefill (the log-prob forward after rollout), against the oracle."""
    rng = np.random.default_rng(11)
    B, hkv, G, d, maxb = 5, 2, 4, 128, 5
    NB = B * maxb + 3
    lens = rng.integers(1, 16 * maxb, B).astype(np.int32)
    table = rng.permutation(NB)[:B * maxb].reshape(B, maxb).astype(np.int32)
    kc = torch.zeros((NB, hkv, 16, d), dtype=torch.uint8, device=DEV)
    vc = torch.zeros((NB, hkv, d, 16), dtype=torch.uint8, device=DEV)
    sc = torch.ones((2, NB, hkv), dtype=torch.float32, device=DEV)
    tdev = torch.from_numpy(table).to(DEV)
    for t in range(int(lens.max())):
        pos = torch.from_numpy(np.where(t < lens, t, -1).astype(np.int32)).to(DEV)
        kn = torch.randn((B, hkv, d), device=DEV).to(torch.bfloat16)
        vn = torch.randn((B, hkv, d), device=DEV).to(torch.bfloat16)
        lib.paged_kv_append(kn, vn, kc, vc, sc, tdev, pos)
    counts = np.maximum(lens // 2, 1).astype(np.int32)
    offs = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    q = torch.randn((int(offs[-1]), hkv * G, d), device=DEV).to(torch.bfloat16)
    out = torch.empty(q.shape, dtype=torch.float32, device=DEV)
    lib.paged_prefill_attention(q, torch.from_numpy(offs).to(DEV), kc, vc, tdev, torch.from_numpy(lens).to(DEV), sc,
                                out, d ** -0.5)
    torch.cuda.synchronize()
    ref = oracle.paged_prefill_attention(q=U.raw(q), q_offsets=offs, k_cache=U.raw(kc), v_cache=U.raw(vc),
                                         block_table=table, seq_lens=lens, softmax_scale=d ** -0.5, q_dtype="bf16",
                                         kv_dtype="fp8_e4m3", kv_scales=U.raw(sc))
    U.assert_close(U.out_to_f64(out), ref, "fp8_e4m3", "append then prefill")
    assert lib.read_device_status() == 0


@pytest.mark.parametrize("name", ["logprob_gqa7b_bf16", "logprob_gqa7b_fp8kv", "chunk512_gqa7b_bf16"])
def test_prefill_full_size_whole_tensor(lib, name):
    """The benchmarked prefills at full size, in the launch the benchmark
    times: the log-prob forward over the 7B GQA step's 64 sequences (every
    token a query, 193,538 rows, 28 / 4 heads; bf16 and fp8 caches) and the
    chunked prefill (each sequence's last 512 tokens, 32,240 rows), compared
    with the oracle over every output element. The oracle runs over slices of
    64 query rows in the worker pool, longest sequences first."""
    w = W.WORKLOADS[name]
    pin = W.generate_prefill(w, DEV)
    print(f"[prefill whole] {name} T={int(pin.q.shape[0])}", flush=True)
    out = run(lib, pin, torch.bfloat16)
    assert lib.read_device_status() == 0
    got = U.out_to_f64(out)
    ref = U.oracle_prefill_whole(pin, name)
    max_abs, rel_l2 = U.assert_close(got, ref, w.kv_dtype, f"{name} whole tensor", bf16_out_rounding=True)
    worst, at = U.worst_row_rel_l2(got, ref)
    print(f"[prefill whole] max_abs {max_abs:.3e} rel_l2 {rel_l2:.3e}; worst row rel_l2 {worst:.3e} at {at}",
          flush=True)
