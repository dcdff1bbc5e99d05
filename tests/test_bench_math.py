"""The byte and flop counts the benchmark's roofline figures rest on, checked
against independent counts on small cases (hand-computed sums, brute-force
enumeration of visible (query, key) pairs)."""

import numpy as np

import bench
from paper_2605_20863_amd import workloads as W


def wl(hq=8, hkv=2, d=64, kv="bf16", q="bf16", q_tokens=1):
    return W.Workload("t", 0, hq, hkv, d, q, kv, ("uniform", 1, 1), cfg_id=0, q_tokens=q_tokens)


def test_decode_bytes_by_hand():
    lens = np.array([17, 0, 32, 1])
    w = wl()
    got, tokens = bench.algorithmic_bytes(w, lens)
    # tokens 50; blocks 2 + 0 + 2 + 1 = 5; K and V of 2 KV heads x 64 dims x 2 bytes per token
    kv = 50 * 2 * 2 * 64 * 2
    q_out = 2 * 4 * 1 * 8 * 64 * 2
    assert tokens == 50
    assert got == kv + q_out + 4 * 5 + 4 * 4


def test_decode_bytes_fp8_scales_and_query_tokens():
    lens = np.array([16, 33])
    w = wl(kv="fp8_e4m3", q_tokens=3)
    got, _ = bench.algorithmic_bytes(w, lens)
    blocks = 1 + 3
    kv = 49 * 2 * 2 * 64 * 1
    scales = blocks * 2 * 2 * 4        # K and V scale per (block, KV head)
    q_out = 2 * 2 * 3 * 8 * 64 * 2
    assert got == kv + scales + q_out + 4 * blocks + 4 * 2


def test_decode_bytes_count_shared_blocks_once():
    lens = np.array([40, 50, 35, 36])          # two groups of two
    shared = (2, np.array([2, 1]))             # group 0 shares 2 blocks, group 1 shares 1
    w = wl()
    plain, tokens = bench.algorithmic_bytes(w, lens)
    uniq, tokens2 = bench.algorithmic_bytes(w, lens, shared)
    assert tokens == tokens2 == 161
    # one copy of each shared block is dropped per extra member: (2 - 1) * (2 + 1) blocks of 16 tokens
    assert plain - uniq == 3 * 16 * 2 * 2 * 64 * 2


def test_prefill_flops_match_brute_force():
    rng = np.random.default_rng(5)
    w = wl(hq=28, hkv=4, d=128)
    for _ in range(20):
        B = int(rng.integers(1, 6))
        lens = rng.integers(0, 90, B)
        counts = np.array([int(rng.integers(0, L + 3)) for L in lens])  # n may exceed L
        flops, pairs = bench.prefill_flops(w, lens, counts)
        brute = 0
        for L, n in zip(lens, counts):
            for i in range(n):
                pos = L - n + i             # query position; it sees keys 0 .. pos that exist
                brute += sum(1 for k in range(L) if k <= pos)
        assert pairs == brute
        assert flops == 4 * 128 * 28 * brute


def test_prefill_flops_full_causal_closed_form():
    w = wl(hq=4, hkv=4, d=64)
    lens = np.array([100, 7])
    _, pairs = bench.prefill_flops(w, lens, lens)     # every token a query: L (L + 1) / 2 pairs
    assert pairs == 100 * 101 // 2 + 7 * 8 // 2


def test_append_bytes_by_hand():
    B = 3
    assert bench.append_bytes(wl(kv="bf16"), B) == 2 * B * 2 * 64 * (2 + 2) + 8 * B
    # fp8: new rows read as bf16, written as codes; K and V scales read and written
    assert bench.append_bytes(wl(kv="fp8_e4m3"), B) == 2 * B * 2 * 64 * (2 + 1) + 2 * 2 * B * 2 * 4 + 8 * B


def test_source_digest_ignores_comments_only(tmp_path):
    a = tmp_path / "a.hip"
    a.write_text("// header\nint f(int x) {  /* twice */ return 2 * x; }\n")
    b = tmp_path / "b.hip"
    b.write_text("// a different header\n\nint f(int x) {\n  return 2 * x;  // doubled\n}\n")
    c = tmp_path / "c.hip"
    c.write_text("// header\nint f(int x) { return 3 * x; }\n")
    assert bench.source_digest(a) == bench.source_digest(b)
    assert bench.source_digest(a) != bench.source_digest(c)
