"""Pins of the varlen prefill oracle, ``oracle.paged_prefill_attention``:
torch fp64 SDPA with an explicit causal mask on the contiguous keys and
values of tests/_cases.py, a pure-Python brute force, and the chunked-prefill
property (prefilling n tokens equals prefilling them in two chunks against the
same cache). Planted mistakes in the window or the packing must fail a pin."""

import math

import numpy as np
import pytest
import torch

import oracle
import oracle.decode_attention as od
from tests import _cases


def _packed_queries(ns, hq, d, dtype, seed):
    rng = np.random.default_rng(seed)
    stored, exact = _cases._store(rng.standard_normal((int(sum(ns)), hq, d)), dtype)
    offs = np.concatenate([[0], np.cumsum(ns)]).astype(np.int32)
    return stored, exact, offs


def _pf(o, case, q, offs, **kw):
    args = case.oracle_args()
    args.update(q=q, q_offsets=offs, **kw)
    return o.paged_prefill_attention(**args)


def _sdpa_causal(case, q64, offs, b, hq, hkv):
    G = hq // hkv
    L = case.K64[b].shape[0]
    r0, r1 = int(offs[b]), int(offs[b + 1])
    n = r1 - r0
    K = torch.from_numpy(case.K64[b]).permute(1, 0, 2).repeat_interleave(G, dim=0).unsqueeze(0)
    V = torch.from_numpy(case.V64[b]).permute(1, 0, 2).repeat_interleave(G, dim=0).unsqueeze(0)
    qq = torch.from_numpy(q64[r0:r1]).permute(1, 0, 2).unsqueeze(0)         # [1, Hq, n, D]
    mask = torch.arange(L)[None, :] <= (L - n + torch.arange(n))[:, None]
    out = torch.nn.functional.scaled_dot_product_attention(qq, K, V, attn_mask=mask, scale=case.softmax_scale)
    out = out[0].permute(1, 0, 2).numpy()
    out[~mask.any(dim=1).numpy()] = 0.0
    return out


def pin_pf_sdpa(o):
    lens = [1, 16, 17, 40, 64, 100]
    for kv in ("f32", "bf16", "fp8_e4m3"):
        for ns, (hq, hkv) in (([1, 16, 17, 40, 64, 100], (4, 4)), ([1, 5, 17, 3, 64, 37], (8, 2)),
                              ([0, 2, 20, 40, 1, 0], (6, 1)), ([3, 18, 1, 45, 70, 101], (2, 2))):
            case = _cases.build(lens, hq, hkv, 16, kv_dtype=kv, seed=500 + hq)
            q, q64, offs = _packed_queries(ns, hq, 16, case.q_dtype, 501 + hkv)
            out = _pf(o, case, q, offs)
            for b in range(len(lens)):
                np.testing.assert_allclose(out[offs[b]:offs[b + 1]], _sdpa_causal(case, q64, offs, b, hq, hkv),
                                           rtol=0, atol=1e-12, err_msg=f"kv={kv} ns={ns} b={b}")


def pin_pf_brute_force(o):
    lens = [3, 19]
    ns = [3, 5]
    case = _cases.build(lens, 2, 1, 4, kv_dtype="f32", seed=510)
    q, q64, offs = _packed_queries(ns, 2, 4, "f32", 511)
    out = _pf(o, case, q, offs)
    for b, L in enumerate(lens):
        for i in range(ns[b]):
            r = offs[b] + i
            m_vis = L - ns[b] + i + 1
            for h in range(2):
                s = [case.softmax_scale * math.fsum(q64[r, h, e] * case.K64[b][t, 0, e] for e in range(4))
                     for t in range(m_vis)]
                m = max(s)
                w = [math.exp(x - m) for x in s]
                ref = [math.fsum(w[t] * case.V64[b][t, 0, e] for t in range(m_vis)) / math.fsum(w) for e in range(4)]
                np.testing.assert_allclose(out[r, h], ref, rtol=0, atol=1e-13)


def pin_pf_chunked(o):
    """Prefilling n tokens in one call equals two chunks: the first n1 tokens
    against a cache of length L - n + n1, then the remaining n - n1 against L."""
    lens = [50, 90]
    ns = [30, 90]
    case = _cases.build(lens, 4, 2, 16, kv_dtype="bf16", seed=520)
    q, _, offs = _packed_queries(ns, 4, 16, "bf16", 521)
    full = _pf(o, case, q, offs)
    for b, (L, n) in enumerate(zip(lens, ns)):
        n1 = n // 3
        r0 = offs[b]
        first = _pf(o, case, q[r0:r0 + n1], np.array([0, n1], np.int32), seq_lens=np.array([L - n + n1], np.int32),
                    block_table=case.block_table[b:b + 1])
        second = _pf(o, case, q[r0 + n1:r0 + n], np.array([0, n - n1], np.int32), seq_lens=np.array([L], np.int32),
                     block_table=case.block_table[b:b + 1])
        np.testing.assert_array_equal(full[r0:r0 + n1], first)
        np.testing.assert_array_equal(full[r0 + n1:r0 + n], second)


PINS = [pin_pf_sdpa, pin_pf_brute_force, pin_pf_chunked]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_prefill_pin(pin):
    pin(oracle)


def _variant(visible=None, pack_shift=0):
    def pf(q, q_offsets, k_cache, v_cache, block_table, seq_lens, softmax_scale, q_dtype, kv_dtype,
           kv_scales=None, seqs=None):
        T, hq, d = q.shape
        hkv = k_cache.shape[1]
        G = hq // hkv
        qd = od.decode(q, q_dtype)
        out = np.zeros((T, hq, d))
        for b in range(len(seq_lens)):
            L = int(seq_lens[b])
            r0, r1 = int(q_offsets[b]), int(q_offsets[b + 1])
            n = r1 - r0
            for g in range(hkv):
                K, V = od.gather_sequence(k_cache, v_cache, block_table, L, b, g, kv_dtype, kv_scales)
                for i in range(n):
                    vis = visible(L, n, i) if visible else L - n + i + 1
                    vis = min(max(vis, 0), L)
                    src = min(max(r0 + i + pack_shift, 0), T - 1)
                    for h in range(g * G, (g + 1) * G):
                        out[r0 + i, h] = od.attend(qd[src, h], K[:vis], V[:vis], softmax_scale)
        return out
    return lambda mp: mp.setattr(oracle, "paged_prefill_attention", pf)


MUTANTS = {
    "window_off_by_one": _variant(visible=lambda L, n, i: L - n + i),
    "window_from_start": _variant(visible=lambda L, n, i: i + 1),
    "non_causal": _variant(visible=lambda L, n, i: L),
    "queries_shifted": _variant(pack_shift=1),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_prefill_mutants_are_caught(name, monkeypatch):
    MUTANTS[name](monkeypatch)
    failed = []
    for pin in PINS:
        try:
            pin(oracle)
        except Exception:  # noqa: BLE001 - any failure counts as caught
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
