"""Seeded generators: determinism, block-table structure and poison placement."""

import numpy as np
import torch

from paper_2605_20863_amd import workloads as W


def test_lengths_follow_the_recipes():
    for name, w in W.WORKLOADS.items():
        lens, prompts = W.sample_lengths(w)
        assert lens.shape == (w.num_seqs,) and lens.dtype == np.int32
        kind = w.lengths[0]
        if kind == "uniform":
            assert lens.min() >= w.lengths[1] and lens.max() <= w.lengths[2]
        elif kind == "lognormal":
            _, med, sigma, lo, hi = w.lengths
            assert lens.min() >= lo and lens.max() <= hi
            # the median of a lognormal sample sits near the recipe's median
            assert 0.7 * med < np.median(lens) < 1.3 * med
        else:
            _, P, S, plo, phi, med, sigma, rmax = w.lengths
            assert prompts.min() >= plo and prompts.max() <= phi
            resp = lens - prompts
            assert resp.min() >= 1 and resp.max() <= rmax
            assert np.all(prompts.reshape(P, S) == prompts.reshape(P, S)[:, :1])


def test_layout_is_deterministic_and_a_permutation():
    w = W.WORKLOADS["gqa7b_bf16"]
    a, b = W.make_layout(w), W.make_layout(w)
    assert np.array_equal(a.block_table, b.block_table) and np.array_equal(a.seq_lens, b.seq_lens)
    used = a.block_table[a.block_table >= 0]
    assert len(np.unique(used)) == len(used)          # no block shared without GRPO
    assert used.max() < a.num_blocks
    assert a.num_blocks - len(used) >= 0.05 * len(used)   # >= 5% spare poisoned blocks
    nblk = (a.seq_lens + 15) // 16
    for r, n in enumerate(nblk):
        assert (a.block_table[r, :n] >= 0).all() and (a.block_table[r, n:] == -1).all()


def test_grpo_groups_share_full_prompt_blocks():
    w = W.SMALL_WORKLOADS["grpo_bf16"]
    lay = W.make_layout(w)
    S = w.lengths[2]
    for g0 in range(0, w.num_seqs, S):
        shared = int(lay.prompt_lens[g0]) // 16
        rows = lay.block_table[g0:g0 + S]
        assert (rows[:, :shared] == rows[:1, :shared]).all()
        priv = [set(r[shared:(int(L) + 15) // 16]) for r, L in zip(rows, lay.seq_lens[g0:g0 + S])]
        for i in range(S):
            for j in range(i + 1, S):
                assert not (priv[i] & priv[j])


def test_values_and_poison():
    w = W.SMALL_WORKLOADS["fp8kv"]
    a = W.generate(w)
    b = W.generate(w)
    assert torch.equal(a.k_cache, b.k_cache)
    assert torch.allclose(a.kv_scales, b.kv_scales, rtol=0, atol=0, equal_nan=True)
    lay = a.layout
    unused = np.nonzero(~lay.used)[0]
    assert (a.k_cache[unused] == 0x7F).all() and torch.isnan(a.kv_scales[:, unused]).all()
    for r, L in enumerate(lay.seq_lens):
        if L % 16:
            p = lay.block_table[r, L // 16]
            assert (a.k_cache[p, :, L % 16:, :] == 0x7F).all()
            assert (a.v_cache[p, :, :, L % 16:] == 0x7F).all()
            assert (a.k_cache[p, :, :L % 16, :] != 0x7F).all()
    # scales map each tile's amax to the largest finite code
    used = np.nonzero(lay.used)[0][:5]
    codes = a.k_cache[used].view(torch.float8_e4m3fn).float().abs()
    codes = torch.where(torch.isnan(codes), torch.zeros_like(codes), codes)
    assert torch.all(codes <= 448) and codes.max() == 448
    t = W.generate(W.SMALL_WORKLOADS["gqa7b_bf16"])
    assert t.k_cache.dtype == torch.bfloat16 and t.v_cache.shape[2:] == (128, 16)


def test_group_prefix_matches_the_shared_blocks():
    """group_prefix reports exactly the leading block ids a GRPO group's samples share."""
    for name in ("grpo_bf16", "grpo_longprompt_bf16"):
        w = W.WORKLOADS[name]
        lay = W.make_layout(w)
        gs, sb = W.group_prefix(w, lay)
        assert gs == w.lengths[2] and sb.shape == (w.num_seqs // gs,)
        for g in range(len(sb)):
            rows = lay.block_table[g * gs:(g + 1) * gs]
            assert (rows[:, :sb[g]] == rows[0, :sb[g]]).all()
            nxt = rows[:, sb[g]]                 # first private block (prompt tail or response)
            assert len(np.unique(nxt[nxt >= 0])) == (nxt >= 0).sum()
    assert W.group_prefix(W.WORKLOADS["gqa7b_bf16"], W.make_layout(W.WORKLOADS["gqa7b_bf16"])) is None
