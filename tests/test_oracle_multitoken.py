"""Pins of the multi-token (speculative verification) oracle,
``oracle.paged_multi_token_attention``, to computations other than itself:
torch's fp64 scaled_dot_product_attention with an explicit causal mask on the
contiguous keys and values that tests/_cases.py scatters into the paged
layout, and a pure-Python brute force on tiny inputs. Planted mistakes in the
causal window (off by one, reversed, ignored) must each fail a pin.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import oracle.decode_attention as od
from tests import _cases


def _queries(B, Q, hq, d, dtype, seed):
    rng = np.random.default_rng(seed)
    stored, exact = _cases._store(rng.standard_normal((B, Q, hq, d)), dtype)
    return stored, exact


def _mt(o, case, q, **kw):
    args = case.oracle_args()
    args.update(q=q, **kw)
    return o.paged_multi_token_attention(**args)


def _sdpa_causal(case, q64, b, hq, hkv):
    """torch fp64 SDPA of sequence b's Q queries; query i sees keys 0 .. L - Q + i."""
    G = hq // hkv
    L = case.K64[b].shape[0]
    Q = q64.shape[1]
    K = torch.from_numpy(case.K64[b]).permute(1, 0, 2).repeat_interleave(G, dim=0).unsqueeze(0)
    V = torch.from_numpy(case.V64[b]).permute(1, 0, 2).repeat_interleave(G, dim=0).unsqueeze(0)
    qq = torch.from_numpy(q64[b]).permute(1, 0, 2).unsqueeze(0)             # [1, Hq, Q, D]
    keys = torch.arange(L)[None, :]
    last = (L - Q + torch.arange(Q))[:, None]
    mask = keys <= last                                                     # [Q, L]
    out = torch.nn.functional.scaled_dot_product_attention(qq, K, V, attn_mask=mask, scale=case.softmax_scale)
    out = out[0].permute(1, 0, 2).numpy()                                   # [Q, Hq, D]
    out[~mask.any(dim=1).numpy()] = 0.0                                     # no visible key -> zeros
    return out


def pin_mt_sdpa(o):
    lens = [1, 3, 4, 15, 16, 17, 33, 64, 90]
    for kv in ("f32", "bf16", "fp8_e4m3"):
        for Q, (hq, hkv) in ((1, (8, 2)), (2, (8, 2)), (4, (4, 4)), (3, (6, 1))):
            case = _cases.build(lens, hq, hkv, 16, kv_dtype=kv, seed=100 + Q + hq)
            q, q64 = _queries(len(lens), Q, hq, 16, case.q_dtype, 200 + Q)
            out = _mt(o, case, q)
            for b in range(len(lens)):
                np.testing.assert_allclose(out[b], _sdpa_causal(case, q64, b, hq, hkv), rtol=0, atol=1e-12,
                                           err_msg=f"kv={kv} Q={Q} b={b}")


def pin_mt_brute_force(o):
    lens = [2, 5, 18]
    case = _cases.build(lens, 2, 1, 4, kv_dtype="f32", seed=300)
    Q = 3
    q, q64 = _queries(len(lens), Q, 2, 4, "f32", 301)
    out = _mt(o, case, q)
    for b, L in enumerate(lens):
        for i in range(Q):
            n = L - Q + i + 1
            for h in range(2):
                if n <= 0:
                    assert not out[b, i, h].any()
                    continue
                s = [case.softmax_scale * math.fsum(q64[b, i, h, e] * case.K64[b][t, 0, e] for e in range(4))
                     for t in range(n)]
                m = max(s)
                w = [math.exp(x - m) for x in s]
                ref = [math.fsum(w[t] * case.V64[b][t, 0, e] for t in range(n)) / math.fsum(w) for e in range(4)]
                np.testing.assert_allclose(out[b, i, h], ref, rtol=0, atol=1e-13)


def pin_mt_last_query_is_decode(o):
    """The last query token sees the whole sequence: it is the one-token decode
    of the same sequence, checked against torch SDPA without a mask."""
    lens = [7, 16, 40]
    case = _cases.build(lens, 4, 2, 16, kv_dtype="bf16", seed=400)
    q, q64 = _queries(len(lens), 4, 4, 16, "bf16", 401)
    out = _mt(o, case, q)
    for b, L in enumerate(lens):
        G = 2
        K = torch.from_numpy(case.K64[b]).permute(1, 0, 2).repeat_interleave(G, dim=0).unsqueeze(0)
        V = torch.from_numpy(case.V64[b]).permute(1, 0, 2).repeat_interleave(G, dim=0).unsqueeze(0)
        qq = torch.from_numpy(q64[b, 3]).unsqueeze(0).unsqueeze(2)
        ref = torch.nn.functional.scaled_dot_product_attention(qq, K, V, scale=case.softmax_scale)[0, :, 0].numpy()
        np.testing.assert_allclose(out[b, 3], ref, rtol=0, atol=1e-12)


PINS = [pin_mt_sdpa, pin_mt_brute_force, pin_mt_last_query_is_decode]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_multitoken_pin(pin):
    pin(oracle)


def _window_variant(visible):
    def mt(q, k_cache, v_cache, block_table, seq_lens, softmax_scale, q_dtype, kv_dtype, kv_scales=None, seqs=None):
        B, Q, hq, d = q.shape
        hkv = k_cache.shape[1]
        G = hq // hkv
        qd = od.decode(q, q_dtype)
        out = np.zeros((B, Q, hq, d))
        for b in range(B):
            L = int(seq_lens[b])
            for g in range(hkv):
                K, V = od.gather_sequence(k_cache, v_cache, block_table, L, b, g, kv_dtype, kv_scales)
                for i in range(Q):
                    n = min(max(visible(L, Q, i), 0), L)
                    for h in range(g * G, (g + 1) * G):
                        out[b, i, h] = od.attend(qd[b, i, h], K[:n], V[:n], softmax_scale)
        return out
    return lambda mp: mp.setattr(oracle, "paged_multi_token_attention", mt)


MUTANTS = {
    "window_off_by_one": _window_variant(lambda L, Q, i: L - Q + i),
    "window_reversed": _window_variant(lambda L, Q, i: L - i),
    "window_ignored": _window_variant(lambda L, Q, i: L),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_multitoken_mutants_are_caught(name, monkeypatch):
    MUTANTS[name](monkeypatch)
    failed = []
    for pin in PINS:
        try:
            pin(oracle)
        except Exception:  # noqa: BLE001 - any failure counts as caught
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
