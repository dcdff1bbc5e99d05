"""Pins of the CPU fp64 oracle against facts that do not come from the oracle.

Each ``pin_*`` function raises AssertionError (or any exception) when the
oracle module passed in disagrees with an independent fact:

* a hand-worked example and hand-derived fp8 codes (tests/golden/);
* exhaustive decoding checks of bf16 and OCP e4m3 against torch's casts;
* torch's fp64 scaled_dot_product_attention on contiguous K/V scattered into
  the paged layout by tests/_cases.py (independent indexing);
* pure-Python brute force (math.exp, math.fsum) over the paged arrays;
* closed forms (one key -> its value; equal keys or a zero scale -> mean of V);
* invariances (block and token permutations, key shifts, linearity in V,
  GQA == MHA with repeated KV heads, power-of-two fp8 scale moves);
* the log-sum-exp split identity, poison that must never be read, empty
  sequences.

``test_mutants_are_caught`` plants plausible mistakes in the oracle (on the
CPU) and checks that every one of them fails at least one pin.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import oracle.decode_attention as od
from tests import _cases

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
DTYPES = ("f32", "bf16", "fp8_e4m3")


def _run(o, case, **kw):
    args = case.oracle_args()
    args.update(kw)
    return o.paged_decode_attention(**args)


# --------------------------------------------------------------------------- pins

def pin_hand_example(o):
    ex = json.load(open(os.path.join(GOLDEN, "hand_example.json")))
    D = len(ex["q"])
    k_cache = np.full((2, 1, 16, D), np.nan, dtype=np.float32)
    v_cache = np.full((2, 1, D, 16), np.nan, dtype=np.float32)
    # store the two tokens in physical block 1 (block 0 is poison)
    for t, (k, v) in enumerate(zip(ex["keys"], ex["values"])):
        k_cache[1, 0, t, :] = k
        v_cache[1, 0, :, t] = v
    out = o.paged_decode_attention(
        q=np.array([[ex["q"]]], dtype=np.float32), k_cache=k_cache, v_cache=v_cache,
        block_table=np.array([[1]], dtype=np.int32), seq_lens=np.array([2], dtype=np.int32),
        softmax_scale=ex["softmax_scale"], q_dtype="f32", kv_dtype="f32")
    # keys were stored in float32: ln 3 rounds, so allow that rounding only
    k1 = float(np.float32(ex["keys"][1][0]))
    w1 = math.exp(k1)
    exact = np.array([4.0 / (1 + w1), 8.0 * w1 / (1 + w1)])
    np.testing.assert_allclose(exact, ex["expected"], atol=1e-6)
    np.testing.assert_allclose(out[0, 0], exact, rtol=0, atol=ex["tolerance"] * 10)


def pin_decoders(o):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    got = o.bf16_to_f64(bits)
    assert np.array_equal(np.isnan(ref), np.isnan(got))
    m = ~np.isnan(ref)
    assert np.array_equal(ref[m], got[m]) and np.array_equal(np.signbit(ref[m]), np.signbit(got[m]))
    codes = np.arange(256, dtype=np.uint8)
    ref8 = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got8 = o.e4m3fn_to_f64(codes)
    assert np.array_equal(np.isnan(ref8), np.isnan(got8))
    m = ~np.isnan(ref8)
    assert np.array_equal(ref8[m], got8[m]) and np.array_equal(np.signbit(ref8[m]), np.signbit(got8[m]))


def pin_e4m3_golden(o):
    g = json.load(open(os.path.join(GOLDEN, "e4m3fn_codes.json")))
    for code, val in g["codes"].items():
        got = float(o.e4m3fn_to_f64(np.array([int(code, 16)], dtype=np.uint8))[0])
        if val == "nan":
            assert math.isnan(got), code
        else:
            assert got == val and math.copysign(1, got) == math.copysign(1, val), (code, got, val)


def _sdpa(case, b, hq, hkv):
    """torch fp64 SDPA on the contiguous K/V of sequence b (KV heads repeated)."""
    G = hq // hkv
    K = torch.from_numpy(case.K64[b]).permute(1, 0, 2)          # [Hkv, L, D]
    V = torch.from_numpy(case.V64[b]).permute(1, 0, 2)
    K = K.repeat_interleave(G, dim=0).unsqueeze(0)              # [1, Hq, L, D]
    V = V.repeat_interleave(G, dim=0).unsqueeze(0)
    q = torch.from_numpy(case.q64[b]).unsqueeze(0).unsqueeze(2)  # [1, Hq, 1, D]
    o = torch.nn.functional.scaled_dot_product_attention(q, K, V, scale=case.softmax_scale)
    return o[0, :, 0, :].numpy()


def pin_sdpa(o):
    lens = [1, 15, 16, 17, 33, 47, 64, 100]
    for kv in DTYPES:
        for (hq, hkv) in ((8, 2), (4, 4), (7, 1)):
            case = _cases.build(lens, hq, hkv, 16, kv_dtype=kv, seed=11 + hq)
            out = _run(o, case)
            for b in range(len(lens)):
                np.testing.assert_allclose(out[b], _sdpa(case, b, hq, hkv), rtol=0, atol=1e-12,
                                           err_msg=f"{kv} hq={hq} hkv={hkv} b={b}")


def _brute(case, hq, hkv):
    """Pure-Python loops over the paged arrays; torch decodes the storage."""
    def dec(a, dtype):
        t = torch.from_numpy(np.ascontiguousarray(a))
        if dtype == "bf16":
            t = t.view(torch.int16).view(torch.bfloat16)
        elif dtype == "fp8_e4m3":
            t = t.view(torch.float8_e4m3fn)
        return t.to(torch.float64).tolist()
    kc, vc = dec(case.k_cache, case.kv_dtype), dec(case.v_cache, case.kv_dtype)
    qv = dec(case.q, case.q_dtype)
    sc = case.kv_scales.astype(np.float64).tolist()
    G = hq // hkv
    B = len(case.seq_lens)
    D = case.q.shape[2]
    out = [[[0.0] * D for _ in range(hq)] for _ in range(B)]
    for b in range(B):
        L = int(case.seq_lens[b])
        for h in range(hq):
            g = h // G
            logits, vals = [], []
            for t in range(L):
                p = int(case.block_table[b][t // 16])
                slot = t % 16
                ks = sc[0][p][g] if case.kv_dtype == "fp8_e4m3" else 1.0
                vs = sc[1][p][g] if case.kv_dtype == "fp8_e4m3" else 1.0
                dot = math.fsum(qv[b][h][d] * (kc[p][g][slot][d] * ks) for d in range(D))
                logits.append(case.softmax_scale * dot)
                vals.append([vc[p][g][d][slot] * vs for d in range(D)])
            if L == 0:
                continue
            mx = max(logits)
            w = [math.exp(s - mx) for s in logits]
            den = math.fsum(w)
            for d in range(D):
                out[b][h][d] = math.fsum(w[t] * vals[t][d] for t in range(L)) / den
    return np.array(out)


def pin_brute_force(o):
    for kv in DTYPES:
        case = _cases.build([0, 1, 5, 16, 18, 40], 4, 2, 8, kv_dtype=kv, seed=5)
        np.testing.assert_allclose(_run(o, case), _brute(case, 4, 2), rtol=0, atol=1e-12, err_msg=kv)


def pin_single_key(o):
    for kv in DTYPES:
        case = _cases.build([1, 1, 1], 6, 3, 16, kv_dtype=kv, seed=3)
        out = _run(o, case)
        for b in range(3):
            for h in range(6):
                assert np.array_equal(out[b, h], case.V64[b][0, h // 2]), (kv, b, h)


def pin_equal_keys(o):
    same = lambda rng, shape: np.broadcast_to(rng.standard_normal(shape[-1]), shape).copy()
    for kv in ("f32", "bf16"):
        case = _cases.build([37, 70], 4, 2, 16, kv_dtype=kv, seed=4, key_fn=same)
        out = _run(o, case)
        for b in range(2):
            for h in range(4):
                np.testing.assert_allclose(out[b, h], case.V64[b][:, h // 2].mean(axis=0),
                                           rtol=0, atol=1e-13)


def pin_zero_scale(o):
    case = _cases.build([29, 50], 4, 1, 16, kv_dtype="bf16", seed=8, softmax_scale=0.0)
    out = _run(o, case)
    for b in range(2):
        np.testing.assert_allclose(out[b], np.broadcast_to(case.V64[b][:, 0].mean(axis=0), (4, 16)),
                                   rtol=0, atol=1e-13)


def pin_block_perm(o):
    lens = [33, 64, 7]
    a = _cases.build(lens, 4, 2, 16, kv_dtype="bf16", seed=21, spare=5)
    NB = a.k_cache.shape[0]
    perm = np.random.default_rng(99).permutation(NB)   # physical id p -> perm[p]
    inv_k = np.empty_like(a.k_cache)
    inv_v = np.empty_like(a.v_cache)
    inv_s = np.empty_like(a.kv_scales)
    inv_k[perm] = a.k_cache
    inv_v[perm] = a.v_cache
    inv_s[:, perm] = a.kv_scales
    table = np.where(a.block_table >= 0, perm[np.maximum(a.block_table, 0)], -1).astype(np.int32)
    out1 = _run(o, a)
    out2 = o.paged_decode_attention(q=a.q, k_cache=inv_k, v_cache=inv_v, block_table=table,
                                    seq_lens=a.seq_lens, softmax_scale=a.softmax_scale,
                                    q_dtype=a.q_dtype, kv_dtype=a.kv_dtype)
    assert np.array_equal(out1, out2)


def pin_token_perm(o):
    lens = [45, 20]
    a = _cases.build(lens, 4, 2, 16, kv_dtype="f32", seed=31, poison=False)
    rng = np.random.default_rng(5)
    perms = [rng.permutation(L) for L in lens]
    K0 = [a.K64[b][perms[b]] for b in range(2)]
    V0 = [a.V64[b][perms[b]] for b in range(2)]
    b2 = _rebuild_f32(a, K0, V0)
    np.testing.assert_allclose(_run(o, a), _run(o, b2), rtol=0, atol=1e-13)


def _rebuild_f32(a, Ks, Vs):
    """Same table/q as case ``a`` (f32) with new contiguous keys/values."""
    k_cache = a.k_cache.copy()
    v_cache = a.v_cache.copy()
    for b, L in enumerate(a.seq_lens):
        for t in range(int(L)):
            p = a.block_table[b, t // 16]
            k_cache[p, :, t % 16, :] = Ks[b][t]
            v_cache[p, :, :, t % 16] = Vs[b][t]
    c = _cases.Case(**{**a.__dict__})
    c.k_cache, c.v_cache = k_cache, v_cache
    c.K64, c.V64 = Ks, Vs
    return c


def pin_key_shift(o):
    # adding the same vector c to every key (of one KV head) shifts every logit of a
    # query by the same amount, which softmax ignores; use dyadic values so the
    # shifted keys stay exact in float32
    dy = lambda rng, shape: rng.integers(-64, 64, size=shape) / 32.0
    a = _cases.build([40, 23], 4, 2, 8, kv_dtype="f32", seed=41, poison=False, key_fn=dy, q_fn=dy)
    c = np.random.default_rng(1).integers(-8, 8, size=(2, 8)) / 4.0
    Ks = [a.K64[b] + c[None, :, :] for b in range(2)]
    b2 = _rebuild_f32(a, Ks, a.V64)
    np.testing.assert_allclose(_run(o, a), _run(o, b2), rtol=0, atol=1e-12)


def pin_linearity(o):
    # dyadic values keep 2 V - W / 2 exact in float32
    dy = lambda rng, shape: rng.integers(-256, 256, size=shape) / 64.0
    a = _cases.build([30, 41], 4, 2, 8, kv_dtype="f32", seed=51, poison=False, value_fn=dy)
    rng = np.random.default_rng(2)
    W = [rng.integers(-256, 256, size=v.shape) / 64.0 for v in a.V64]
    A = [2.0 * a.V64[b] - 0.5 * W[b] for b in range(2)]
    assert all(np.array_equal(x.astype(np.float32).astype(np.float64), x) for x in A)
    cw = _rebuild_f32(a, a.K64, W)
    ca = _rebuild_f32(a, a.K64, A)
    np.testing.assert_allclose(_run(o, ca), 2.0 * _run(o, a) - 0.5 * _run(o, cw), rtol=0, atol=1e-12)


def pin_gqa_mha(o):
    lens = [19, 48]
    a = _cases.build(lens, 8, 2, 16, kv_dtype="bf16", seed=61)
    G = 4
    k_rep = np.repeat(a.k_cache, G, axis=1)   # KV head g -> heads g*G .. g*G+G-1
    v_rep = np.repeat(a.v_cache, G, axis=1)
    out_gqa = _run(o, a)
    out_mha = o.paged_decode_attention(q=a.q, k_cache=k_rep, v_cache=v_rep, block_table=a.block_table,
                                       seq_lens=a.seq_lens, softmax_scale=a.softmax_scale,
                                       q_dtype=a.q_dtype, kv_dtype=a.kv_dtype)
    assert np.array_equal(out_gqa, out_mha)


def pin_split_lse(o):
    rng = np.random.default_rng(7)
    for L in (1, 2, 17, 100):
        q = rng.standard_normal(16)
        K = rng.standard_normal((L, 16)) * 3
        V = rng.standard_normal((L, 16))
        whole = o.attend(q, K, V, 0.25)
        for _ in range(5):
            cuts = np.sort(rng.integers(0, L + 1, size=rng.integers(1, 5)))
            edges = [0] + list(cuts) + [L]
            parts = [o.attend_partial(q, K[a:b], V[a:b], 0.25) for a, b in zip(edges[:-1], edges[1:])]
            np.testing.assert_allclose(o.combine_partials(parts), whole, rtol=0, atol=1e-12)
        # a partial's (m, l, acc) is itself exact: acc / l is the subset's attention
        m, l, acc = o.attend_partial(q, K, V, 0.25)
        np.testing.assert_allclose(acc / l, whole, rtol=0, atol=1e-13)
        assert m == pytest.approx(np.max(0.25 * (K @ q)), abs=0)


def pin_fp8_pow2(o):
    # doubling every stored code (exact for finite codes up to 224) while halving
    # the scales (exact in binary floating point) must leave the output unchanged
    a = _cases.build([35, 16], 4, 2, 16, kv_dtype="fp8_e4m3", seed=71, fp8_headroom=2.5)
    kv = torch.from_numpy(a.k_cache).view(torch.float8_e4m3fn).to(torch.float64)
    vv = torch.from_numpy(a.v_cache).view(torch.float8_e4m3fn).to(torch.float64)
    finite_max = max(kv[torch.isfinite(kv)].abs().max().item(), vv[torch.isfinite(vv)].abs().max().item())
    assert finite_max <= 224
    c = _cases.Case(**{**a.__dict__})
    c.k_cache = (kv * 2).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    c.v_cache = (vv * 2).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    c.kv_scales = a.kv_scales / 2
    assert not np.array_equal(c.k_cache, a.k_cache)
    assert np.array_equal(_run(o, a), _run(o, c))


def pin_poison(o):
    lens = [3, 17, 32, 50]
    clean = _cases.build(lens, 4, 2, 16, kv_dtype="bf16", seed=81, poison=False)
    dirty = _cases.build(lens, 4, 2, 16, kv_dtype="bf16", seed=81, poison=True)
    out_d = _run(o, dirty)
    assert np.isfinite(out_d).all()
    assert np.array_equal(_run(o, clean), out_d)
    for kv in ("f32", "fp8_e4m3"):
        d = _cases.build(lens, 4, 2, 16, kv_dtype=kv, seed=82, poison=True)
        assert np.isfinite(_run(o, d)).all()


def pin_empty(o):
    a = _cases.build([0, 5, 0], 4, 2, 16, kv_dtype="bf16", seed=91)
    out = _run(o, a)
    assert np.array_equal(out[0], np.zeros((4, 16))) and np.array_equal(out[2], np.zeros((4, 16)))
    np.testing.assert_allclose(out[1], _sdpa(a, 1, 4, 2), rtol=0, atol=1e-12)


PINS = [pin_hand_example, pin_decoders, pin_e4m3_golden, pin_sdpa, pin_brute_force,
        pin_single_key, pin_equal_keys, pin_zero_scale, pin_block_perm, pin_token_perm,
        pin_key_shift, pin_linearity, pin_gqa_mha, pin_split_lse, pin_fp8_pow2, pin_poison,
        pin_empty]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin(oracle)


# ----------------------------------------------------------------- planted mistakes

def _mut_dropped_scale(mp):
    orig = od.attend
    mp.setattr(od, "attend", lambda q, K, V, s: orig(q, K, V, 1.0))


def _mut_exp_sign(mp):
    def bad(q, K, V, scale):
        if K.shape[0] == 0:
            return np.zeros(V.shape[1])
        s = scale * (K @ q)
        w = np.exp(np.max(s) - s)
        return (w @ V) / np.sum(w)
    mp.setattr(od, "attend", bad)


def _mut_count_norm(mp):
    def bad(q, K, V, scale):
        if K.shape[0] == 0:
            return np.zeros(V.shape[1])
        s = scale * (K @ q)
        w = np.exp(s - np.max(s))
        return (w @ V) / len(w)
    mp.setattr(od, "attend", bad)


def _mut_head_modulo(mp):
    def bad(q, k_cache, v_cache, block_table, seq_lens, softmax_scale, q_dtype, kv_dtype,
            kv_scales=None, seqs=None):
        B, hq, d = q.shape
        hkv = k_cache.shape[1]
        qd = od.decode(q, q_dtype)
        out = np.zeros((B, hq, d))
        for b in range(B):
            for h in range(hq):
                K, V = od.gather_sequence(k_cache, v_cache, block_table, seq_lens[b], b, h % hkv,
                                          kv_dtype, kv_scales)
                out[b, h] = od.attend(qd[b, h], K, V, softmax_scale)
        return out
    mp.setattr(od, "paged_decode_attention", bad)
    mp.setattr(oracle, "paged_decode_attention", bad)


def _gather_variant(k_slot=lambda s, n: s, v_from_k_layout=False, swap_scales=False, drop_v_scale=False):
    def gather(k_cache, v_cache, block_table, seq_len, b, g, kv_dtype, kv_scales=None):
        L = int(seq_len)
        nb, hkv, bs, d = k_cache.shape
        K = np.zeros((L, d))
        V = np.zeros((L, d))
        for t in range(0, L, bs):
            p = int(block_table[b, t // bs])
            n = min(bs, L - t)
            idx = np.array([k_slot(s, n) for s in range(n)])
            kt = od.decode(k_cache[p, g, idx, :], kv_dtype)
            if v_from_k_layout:
                vt = od.decode(v_cache[p, g, :n, :].reshape(-1)[: n * d].reshape(n, d), kv_dtype)
            else:
                vt = od.decode(v_cache[p, g, :, :n], kv_dtype).T
            if kv_dtype == "fp8_e4m3":
                ks, vs = kv_scales[0, p, g], kv_scales[1, p, g]
                if swap_scales:
                    ks, vs = vs, ks
                kt = kt * ks
                vt = vt if drop_v_scale else vt * vs
            K[t:t + n] = kt
            V[t:t + n] = vt
        return K, V
    return gather


def _mut_gather(**kw):
    return lambda mp: mp.setattr(od, "gather_sequence", _gather_variant(**kw))


def _mut_bf16_as_fp16(mp):
    mp.setattr(od, "bf16_to_f64", lambda bits: np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64))
    mp.setattr(oracle, "bf16_to_f64", od.bf16_to_f64)


def _mut_e4m3_bias8(mp):
    def val(c):
        s, e, m = (c >> 7) & 1, (c >> 3) & 0xF, c & 7
        sign = -1.0 if s else 1.0
        if c == 0x80:
            return float("nan")
        if e == 0:
            return sign * math.ldexp(m / 8.0, 1 - 8)
        return sign * math.ldexp(1 + m / 8.0, e - 8)
    table = np.array([val(c) for c in range(256)])
    bad = lambda codes: table[np.asarray(codes, dtype=np.uint8)]
    mp.setattr(od, "e4m3fn_to_f64", bad)
    mp.setattr(oracle, "e4m3fn_to_f64", bad)


def _mut_combine_no_rescale(mp):
    def bad(parts):
        live = [(m, l, a) for (m, l, a) in parts if m != -math.inf]
        if not live:
            return np.zeros_like(parts[0][2])
        return sum(a for _, _, a in live) / sum(l for _, l, _ in live)
    mp.setattr(od, "combine_partials", bad)
    mp.setattr(oracle, "combine_partials", bad)


MUTANTS = {
    "dropped_softmax_scale": _mut_dropped_scale,
    "exp_sign_flipped": _mut_exp_sign,
    "normalise_by_count": _mut_count_norm,
    "head_map_modulo": _mut_head_modulo,
    "k_slots_reversed": _mut_gather(k_slot=lambda s, n: n - 1 - s),
    "v_read_token_major": _mut_gather(v_from_k_layout=True),
    "fp8_scales_swapped": _mut_gather(swap_scales=True),
    "fp8_v_scale_dropped": _mut_gather(drop_v_scale=True),
    "bf16_decoded_as_fp16": _mut_bf16_as_fp16,
    "e4m3_bias_8_fnuz": _mut_e4m3_bias8,
    "combine_without_rescale": _mut_combine_no_rescale,
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutants_are_caught(name, monkeypatch):
    MUTANTS[name](monkeypatch)
    failed = []
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin(oracle)
        except Exception:  # noqa: BLE001 - any failure counts as caught
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
