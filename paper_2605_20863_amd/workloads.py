"""Seeded synthetic decode-step and prefill inputs.

This module draws the inputs of one batched paged-KV decode step: sequence
lengths, block tables, queries and the paged K/V cache (with fp8 encoding and
scales where asked), and the packed queries of a prefill over such a cache. It holds none of the attention arithmetic; both the HIP
path and the CPU oracle consume what it produces.

The paper's workload (a proprietary maths dataset decoded by Qwen2.5-7B,
Qwen3-30B-A3B and Qwen3-235B-A22B, Sec. 6.1) is not available, so these
generators stand in for the decode shapes of its rollout phase: long-tailed
response lengths (Sec. 2.2), GRPO groups that share a prompt (Sec. 2.3,
Sec. 6.3) and the 7B model's 28 query / 4 KV heads (Sec. 6.1).

Cache layout (the paper prescribes none):
    k_cache [NB, Hkv, BS, D]  token-major tile per (block, KV head)
    v_cache [NB, Hkv, D, BS]  dim-major tile per (block, KV head)
    kv_scales [2, NB, Hkv]    fp32 dequant scales (K, V), fp8 caches only

Every physical block not referenced by any sequence, every cache slot past a
sequence's length in its last block and every unused block-table entry holds
poison (NaN data, NaN scales, block id -1): a correct kernel never reads them.
"""

from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np
import torch

SEED = 260520863
BLOCK_SIZE = 16
FP8_MAX = 448.0
_CHUNK_BLOCKS = 4096

_BF16_NAN = 0x7FC0
_FP8_NAN = 0x7F


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and distribution of one decode step.

    ``lengths`` is one of
        ("uniform", lo, hi)                     L ~ U{lo..hi}
        ("lognormal", median, sigma, lo, hi)    L = clip(rint(exp(N(ln median, sigma^2))), lo, hi)
        ("grpo", prompts, samples, plo, phi, median, sigma, rmax)
            groups of ``samples`` sequences share a prompt of length U{plo..phi};
            each sample adds a response of length clip(rint(lognormal), 1, rmax);
            the prompt's full blocks are shared by the whole group.
    """

    name: str
    num_seqs: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    q_dtype: str
    kv_dtype: str
    lengths: tuple
    cfg_id: int
    block_size: int = BLOCK_SIZE
    q_tokens: int = 1      # query tokens per sequence (> 1: q is [B, q_tokens, Hq, D])
    # > 0: a prefill (log-prob forward) whose sequence b has n_b =
    # clip(rint(prefill_frac * L_b), 1, L_b) packed query tokens, its last n_b
    prefill_frac: float = 0.0
    # > 0: a chunked prefill instead, n_b = min(prefill_chunk, L_b): each
    # sequence's last chunk of new tokens attends over its whole cache
    prefill_chunk: int = 0

    @property
    def is_prefill(self) -> bool:
        return self.prefill_frac > 0 or self.prefill_chunk > 0

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # Tiny MHA step, fp32 end to end.
    "tiny_mha_f32": Workload("tiny_mha_f32", 4, 4, 4, 64, "f32", "f32",
                             ("uniform", 1, 256), cfg_id=0),
    # 7B-class GQA step: 28 query / 4 KV heads, bf16.
    "gqa7b_bf16": Workload("gqa7b_bf16", 64, 28, 4, 128, "bf16", "bf16",
                           ("lognormal", 2048, 0.8, 64, 16384), cfg_id=1),
    # The attention shapes of the paper's two larger models (Sec. 6.1): 32 / 4
    # heads (Qwen3-30B-A3B) and 64 / 4 heads (Qwen3-235B-A22B, G = 16 fills
    # every MFMA column), head_dim 128, at the 7B step's lengths (same seeds),
    # so the KV bytes equal the 7B step's and only G differs.
    "qwen30b_bf16": Workload("qwen30b_bf16", 64, 32, 4, 128, "bf16", "bf16",
                             ("lognormal", 2048, 0.8, 64, 16384), cfg_id=1),
    "qwen235b_bf16": Workload("qwen235b_bf16", 64, 64, 4, 128, "bf16", "bf16",
                              ("lognormal", 2048, 0.8, 64, 16384), cfg_id=1),
    # RLVR rollout batch: 32 prompts x 8 GRPO samples sharing prompt blocks.
    "grpo_bf16": Workload("grpo_bf16", 256, 32, 8, 128, "bf16", "bf16",
                          ("grpo", 32, 8, 256, 1024, 4096, 1.0, 32768), cfg_id=2),
    # Long-tail straggler phase: few sequences, 24k-32k tokens each.
    "straggler_bf16": Workload("straggler_bf16", 16, 64, 8, 128, "bf16", "bf16",
                               ("uniform", 24576, 32768), cfg_id=3),
    # fp8 (OCP e4m3) KV cache at scale with per-(block, KV head) scales.
    "fp8kv": Workload("fp8kv", 512, 64, 8, 128, "bf16", "fp8_e4m3",
                      ("lognormal", 8192, 0.9, 128, 65536), cfg_id=4),
    # One GPU's share of the fp8 step under 8-way tensor parallelism over KV
    # heads (rollout TP 8): the same sequences and lengths, 1 KV head and its
    # 8 query heads.
    "fp8kv_tp8": Workload("fp8kv_tp8", 512, 8, 1, 128, "bf16", "fp8_e4m3",
                          ("lognormal", 8192, 0.9, 128, 65536), cfg_id=4),
    # GRPO groups over long shared contexts (3-6k-token prompts, ~1k-token
    # responses): the shape where reading shared blocks once matters most.
    "grpo_longprompt_bf16": Workload("grpo_longprompt_bf16", 256, 32, 8, 128, "bf16", "bf16",
                                     ("grpo", 32, 8, 3072, 6144, 1024, 0.8, 8192), cfg_id=5),
    # Log-prob forward (the compute_log_prob phase) over the 7B GQA step's 64
    # sequences: every token of every sequence is a query, causal over its
    # sequence (~180k packed tokens).
    "logprob_gqa7b_bf16": Workload("logprob_gqa7b_bf16", 64, 28, 4, 128, "bf16", "bf16",
                                   ("lognormal", 2048, 0.8, 64, 16384), cfg_id=1, prefill_frac=1.0),
    # The same log-prob forward over an fp8 (e4m3) cache with per-tile scales.
    "logprob_gqa7b_fp8kv": Workload("logprob_gqa7b_fp8kv", 64, 28, 4, 128, "bf16", "fp8_e4m3",
                                    ("lognormal", 2048, 0.8, 64, 16384), cfg_id=1, prefill_frac=1.0),
    # Chunked prefill over the 7B GQA step's caches: each sequence's last 512
    # tokens (all of a shorter one) attend causally over its whole cache.
    "chunk512_gqa7b_bf16": Workload("chunk512_gqa7b_bf16", 64, 28, 4, 128, "bf16", "bf16",
                                    ("lognormal", 2048, 0.8, 64, 16384), cfg_id=1, prefill_chunk=512),
    # Speculative verification on the 7B GQA step: 2 query tokens per sequence
    # (the drafted one and the next), 14 of the 16 MFMA columns.
    "spec2_gqa7b_bf16": Workload("spec2_gqa7b_bf16", 64, 28, 4, 128, "bf16", "bf16",
                                 ("lognormal", 2048, 0.8, 64, 16384), cfg_id=1, q_tokens=2),
    # 4 query tokens (three drafted): 28 columns, the two-tile MFMA body
    "spec4_gqa7b_bf16": Workload("spec4_gqa7b_bf16", 64, 28, 4, 128, "bf16", "bf16",
                                 ("lognormal", 2048, 0.8, 64, 16384), cfg_id=1, q_tokens=4),
}

# Reduced versions with the same heads, dtypes and length structure, sized so the
# oracle finishes in seconds while still spanning many blocks and split-K
# partitions with ragged tails.
SMALL_WORKLOADS = {
    "tiny_mha_f32": WORKLOADS["tiny_mha_f32"],
    "gqa7b_bf16": WORKLOADS["gqa7b_bf16"].replace(
        name="gqa7b_bf16_small", num_seqs=8, lengths=("lognormal", 600, 0.8, 64, 3000)),
    "grpo_bf16": WORKLOADS["grpo_bf16"].replace(
        name="grpo_bf16_small", num_seqs=16, lengths=("grpo", 2, 8, 40, 200, 300, 1.0, 1500)),
    "straggler_bf16": WORKLOADS["straggler_bf16"].replace(
        name="straggler_bf16_small", num_seqs=2, lengths=("uniform", 2400, 3300)),
    "fp8kv": WORKLOADS["fp8kv"].replace(
        name="fp8kv_small", num_seqs=6, lengths=("lognormal", 500, 0.9, 128, 4000)),
}


def _seed_seq(w: Workload, *key: int) -> np.random.SeedSequence:
    return np.random.SeedSequence(entropy=SEED, spawn_key=(w.cfg_id,) + tuple(key))


def _torch_seed(w: Workload, *key: int) -> int:
    return int(_seed_seq(w, *key).generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


_STREAM_LENGTHS, _STREAM_TABLE, _STREAM_Q, _STREAM_K, _STREAM_V = 0, 1, 2, 3, 4


@dataclasses.dataclass
class Layout:
    """Host-side description of which physical blocks hold which tokens."""

    seq_lens: np.ndarray          # [B] int32
    block_table: np.ndarray       # [B, max_blocks] int32, -1 past the last used block
    num_blocks: int               # NB (includes spare poisoned blocks)
    used: np.ndarray              # [NB] bool: referenced by some sequence
    prompt_lens: Optional[np.ndarray] = None   # [B] for GRPO workloads
    # GRPO: (sample_first_private_block, group_leader_first_private_block, ntok)
    prompt_tail_copies: Optional[list] = None

    @property
    def max_blocks(self) -> int:
        return self.block_table.shape[1]

    @property
    def max_seq_len(self) -> int:
        return int(self.seq_lens.max()) if self.seq_lens.size else 0


def sample_lengths(w: Workload):
    """Sequence lengths (and GRPO prompt lengths) for workload ``w``."""
    rng = np.random.default_rng(_seed_seq(w, _STREAM_LENGTHS))
    kind = w.lengths[0]
    if kind == "uniform":
        _, lo, hi = w.lengths
        return rng.integers(lo, hi + 1, size=w.num_seqs).astype(np.int32), None
    if kind == "lognormal":
        _, median, sigma, lo, hi = w.lengths
        x = np.exp(rng.normal(math.log(median), sigma, size=w.num_seqs))
        return np.clip(np.rint(x), lo, hi).astype(np.int32), None
    if kind == "grpo":
        _, prompts, samples, plo, phi, median, sigma, rmax = w.lengths
        if prompts * samples != w.num_seqs:
            raise ValueError("GRPO workload needs num_seqs == prompts * samples")
        plen = rng.integers(plo, phi + 1, size=prompts)
        resp = np.clip(np.rint(np.exp(rng.normal(math.log(median), sigma, size=w.num_seqs))), 1, rmax)
        prompt_lens = np.repeat(plen, samples).astype(np.int32)
        return (prompt_lens + resp).astype(np.int32), prompt_lens
    raise ValueError(f"unknown length distribution {kind!r}")


def make_layout(w: Workload, seq_lens=None) -> Layout:
    """Assign physical blocks: a seeded random permutation with >= 5% spare blocks.

    For GRPO workloads the full blocks of each prompt are stored once and
    referenced by all samples of the group; the prompt's partial last block is
    duplicated into each sample's first private block.
    """
    bs = w.block_size
    lens, prompt_lens = sample_lengths(w)
    if seq_lens is not None:
        lens = np.asarray(seq_lens, dtype=np.int32)
        prompt_lens = None
    B = lens.shape[0]
    nblk = (lens.astype(np.int64) + bs - 1) // bs
    max_blocks = max(1, int(nblk.max()) if B else 1)
    rng = np.random.default_rng(_seed_seq(w, _STREAM_TABLE))

    # Logical -> "virtual" block numbering, then a random permutation to physical ids.
    table_virtual = np.full((B, max_blocks), -1, dtype=np.int64)
    copies = []
    nvirt = 0
    if prompt_lens is not None:
        samples = w.lengths[2]
        for g0 in range(0, B, samples):
            shared = int(prompt_lens[g0]) // bs
            shared_ids = np.arange(nvirt, nvirt + shared)
            nvirt += shared
            leader_first_private = None
            for b in range(g0, g0 + samples):
                priv = int(nblk[b]) - shared
                table_virtual[b, :shared] = shared_ids
                table_virtual[b, shared:shared + priv] = np.arange(nvirt, nvirt + priv)
                tail = int(prompt_lens[b]) % bs
                if tail and priv > 0:
                    if leader_first_private is None:
                        leader_first_private = nvirt
                    elif nvirt != leader_first_private:
                        copies.append((nvirt, leader_first_private, tail))
                nvirt += priv
    else:
        for b in range(B):
            n = int(nblk[b])
            table_virtual[b, :n] = np.arange(nvirt, nvirt + n)
            nvirt += n
    spare = max(1, int(math.ceil(0.05 * nvirt)))
    NB = nvirt + spare
    perm = rng.permutation(NB)
    table = np.where(table_virtual >= 0, perm[np.maximum(table_virtual, 0)], -1).astype(np.int32)
    used = np.zeros(NB, dtype=bool)
    used[perm[:nvirt]] = True
    copies_phys = [(int(perm[a]), int(perm[b]), n) for (a, b, n) in copies]
    return Layout(lens, table, NB, used, prompt_lens, copies_phys)


def group_prefix(w: Workload, layout: Layout):
    """For a GRPO workload: (group_size, shared_blocks) with shared_blocks[g]
    the number of leading full blocks (the prompt's) that the block tables of
    group g's samples share. None for other workloads."""
    if w.lengths[0] != "grpo" or layout.prompt_lens is None:
        return None
    samples = int(w.lengths[2])
    return samples, (layout.prompt_lens[::samples] // w.block_size).astype(np.int32)


def prefill_counts(w: Workload, seq_lens) -> np.ndarray:
    """Query tokens per sequence of a prefill workload: its last n_b tokens."""
    L = np.asarray(seq_lens, dtype=np.int64)
    if w.prefill_chunk > 0:
        return np.minimum(L, w.prefill_chunk).astype(np.int32)
    n = np.clip(np.rint(w.prefill_frac * L), 1, np.maximum(L, 1))
    return np.where(L > 0, n, 0).astype(np.int32)


@dataclasses.dataclass
class DecodeInputs:
    """Device tensors of one decode step plus its host-side layout."""

    workload: Workload
    layout: Layout
    q: torch.Tensor               # [B, Hq, D] float32 | bfloat16
    k_cache: torch.Tensor         # [NB, Hkv, BS, D] float32 | bfloat16 | uint8 (e4m3fn codes)
    v_cache: torch.Tensor         # [NB, Hkv, D, BS] same dtype as k_cache
    block_table: torch.Tensor     # [B, max_blocks] int32
    seq_lens: torch.Tensor        # [B] int32
    kv_scales: Optional[torch.Tensor]  # [2, NB, Hkv] float32 or None
    softmax_scale: float

    @property
    def device(self):
        return self.q.device


_TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


def _encode(x: torch.Tensor, dtype: str):
    """Store float32 values as ``dtype``; fp8 returns (codes, per-tile scales)."""
    if dtype in _TORCH_DTYPE:
        return x.to(_TORCH_DTYPE[dtype]), None
    if dtype == "fp8_e4m3":
        # One scale per (block, KV head) tile: amax maps to the largest finite code.
        amax = x.abs().amax(dim=(2, 3))
        scale = torch.clamp(amax / FP8_MAX, min=2.0 ** -126)
        y = torch.clamp(x / scale[:, :, None, None], -FP8_MAX, FP8_MAX)
        return y.to(torch.float8_e4m3fn).view(torch.uint8), scale.to(torch.float32)
    raise ValueError(dtype)


def _poison_value(dtype: str, like: torch.Tensor):
    if dtype == "f32":
        return float("nan")
    if dtype == "bf16":
        return torch.tensor(_BF16_NAN, dtype=torch.int16).view(torch.bfloat16).item()
    return _FP8_NAN


def generate(w: Workload, device="cpu", seq_lens=None, q_scale: float = 1.0) -> DecodeInputs:
    """Draw one decode step of workload ``w`` on ``device``.

    q, K and V are i.i.d. N(0, 1) (times ``q_scale`` for q), rounded to the
    storage dtype (round-to-nearest-even; fp8 after per-tile scaling with
    saturation at +-448). Values of physical block p depend only on (workload,
    p), drawn in fixed chunks of physical ids, so any block can be regenerated.
    """
    device = torch.device(device)
    lay = make_layout(w, seq_lens)
    B, hq, hkv, d, bs = lay.seq_lens.shape[0], w.num_q_heads, w.num_kv_heads, w.head_dim, w.block_size
    NB = lay.num_blocks

    gq = torch.Generator(device=device).manual_seed(_torch_seed(w, _STREAM_Q))
    qshape = (B, hq, d) if w.q_tokens == 1 else (B, w.q_tokens, hq, d)
    q = (torch.randn(qshape, generator=gq, device=device, dtype=torch.float32) * q_scale)
    q = q.to(_TORCH_DTYPE[w.q_dtype])

    store = torch.uint8 if w.kv_dtype == "fp8_e4m3" else _TORCH_DTYPE[w.kv_dtype]
    k_cache = torch.empty((NB, hkv, bs, d), dtype=store, device=device)
    v_cache = torch.empty((NB, hkv, d, bs), dtype=store, device=device)
    kv_scales = (torch.empty((2, NB, hkv), dtype=torch.float32, device=device)
                 if w.kv_dtype == "fp8_e4m3" else None)
    for c0 in range(0, NB, _CHUNK_BLOCKS):
        n = min(_CHUNK_BLOCKS, NB - c0)
        chunk = c0 // _CHUNK_BLOCKS
        gk = torch.Generator(device=device).manual_seed(_torch_seed(w, _STREAM_K, chunk))
        gv = torch.Generator(device=device).manual_seed(_torch_seed(w, _STREAM_V, chunk))
        kx = torch.randn((n, hkv, bs, d), generator=gk, device=device, dtype=torch.float32)
        vx = torch.randn((n, hkv, d, bs), generator=gv, device=device, dtype=torch.float32)
        kc, ks = _encode(kx, w.kv_dtype)
        vc, vs = _encode(vx, w.kv_dtype)
        k_cache[c0:c0 + n] = kc
        v_cache[c0:c0 + n] = vc
        if kv_scales is not None:
            kv_scales[0, c0:c0 + n] = ks
            kv_scales[1, c0:c0 + n] = vs
        del kx, vx, kc, vc

    # GRPO: the prompt's partial last block holds the same stored codes in every
    # sample of a group (for fp8 caches each tile keeps its own scale).
    for dst, src, ntok in (lay.prompt_tail_copies or []):
        k_cache[dst, :, :ntok, :] = k_cache[src, :, :ntok, :]
        v_cache[dst, :, :, :ntok] = v_cache[src, :, :, :ntok]

    # Poison: unreferenced blocks and slots past each sequence's end.
    poison = _poison_value(w.kv_dtype, k_cache)
    unused = torch.from_numpy(np.nonzero(~lay.used)[0]).to(device)
    if unused.numel():
        k_cache[unused] = poison
        v_cache[unused] = poison
        if kv_scales is not None:
            kv_scales[:, unused] = float("nan")
    for b in range(B):
        L = int(lay.seq_lens[b])
        if L % bs:
            p = int(lay.block_table[b, L // bs])
            k_cache[p, :, L % bs:, :] = poison
            v_cache[p, :, :, L % bs:] = poison

    return DecodeInputs(
        workload=w,
        layout=lay,
        q=q,
        k_cache=k_cache,
        v_cache=v_cache,
        block_table=torch.from_numpy(lay.block_table).to(device),
        seq_lens=torch.from_numpy(lay.seq_lens).to(device),
        kv_scales=kv_scales,
        softmax_scale=w.softmax_scale,
    )


@dataclasses.dataclass
class PrefillInputs:
    """Packed queries of a prefill over the paged cache of ``cache``."""

    cache: DecodeInputs           # the paged cache, block table and lengths (its q is unused)
    q: torch.Tensor               # [T, Hq, D] bfloat16
    q_offsets: torch.Tensor       # [B + 1] int32 on the device
    offsets: np.ndarray           # the same offsets on the host
    counts: np.ndarray            # [B] query tokens per sequence


def generate_prefill(w: Workload, device="cpu", seq_lens=None, q_counts=None, q_scale: float = 1.0) -> PrefillInputs:
    """Draw a prefill of workload ``w``: the paged cache as ``generate`` draws
    it, and for sequence b the queries of its last ``q_counts[b]`` tokens
    (default ``prefill_counts``), packed in sequence order, i.i.d. N(0, 1)
    times ``q_scale``, rounded to bf16."""
    cache = generate(w, device, seq_lens=seq_lens)
    lens = cache.layout.seq_lens
    counts = prefill_counts(w, lens) if q_counts is None else np.asarray(q_counts, dtype=np.int32)
    if counts.shape != lens.shape:
        raise ValueError("q_counts needs one entry per sequence")
    offsets = np.concatenate([[0], np.cumsum(counts, dtype=np.int64)]).astype(np.int32)
    T = int(offsets[-1])
    device = torch.device(device)
    g = torch.Generator(device=device).manual_seed(_torch_seed(w, _STREAM_Q, 1))
    q = (torch.randn((T, w.num_q_heads, w.head_dim), generator=g, device=device, dtype=torch.float32) * q_scale)
    return PrefillInputs(cache=cache, q=q.to(torch.bfloat16), q_offsets=torch.from_numpy(offsets).to(device),
                         offsets=offsets, counts=counts)
