"""Helpers that hand device inputs to the CPU oracle and compare results.

Only data movement lives here (device -> host copies, raw-bit views, and the
extraction of a few sequences' blocks into a compact cache). No attention
arithmetic: the expected values always come from ``oracle``.
"""

import numpy as np
import torch

import oracle

TOL = {
    # max-abs and relative-L2 bounds per KV dtype
    "f32": (1e-5, None),
    "bf16": (1e-2, 5e-3),
    "fp8_e4m3": (1e-2, 5e-3),
}


def raw(t: torch.Tensor) -> np.ndarray:
    """Stored bits of a tensor as numpy (bf16 -> uint16, fp8 -> uint8)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.float8_e4m3fn:
        return t.view(torch.uint8).numpy()
    return t.numpy()


def out_to_f64(out: torch.Tensor) -> np.ndarray:
    return out.detach().cpu().to(torch.float64).numpy()


def oracle_for(inp, seqs=None):
    """Oracle output [len(seqs), Hq, D] for sequences ``seqs`` of DecodeInputs ``inp``.

    When ``seqs`` is given, only those sequences' physical blocks are copied to
    the host (remapped into a compact cache), so full-size workloads can be
    checked on a sample.
    """
    w = inp.workload
    lay = inp.layout
    if seqs is None:
        return oracle.paged_decode_attention(
            q=raw(inp.q), k_cache=raw(inp.k_cache), v_cache=raw(inp.v_cache),
            block_table=lay.block_table, seq_lens=lay.seq_lens, softmax_scale=inp.softmax_scale,
            q_dtype=w.q_dtype, kv_dtype=w.kv_dtype,
            kv_scales=raw(inp.kv_scales) if inp.kv_scales is not None else None)
    seqs = list(seqs)
    nblk = [(int(lay.seq_lens[b]) + 15) // 16 for b in seqs]
    phys = np.unique(np.concatenate([lay.block_table[b, :n] for b, n in zip(seqs, nblk)] + [np.zeros(0, np.int32)]))
    if phys.size == 0:
        phys = np.array([0], dtype=np.int64)
    remap = {int(p): i for i, p in enumerate(phys)}
    idx = torch.from_numpy(phys.astype(np.int64)).to(inp.device)
    kc = raw(inp.k_cache.index_select(0, idx))
    vc = raw(inp.v_cache.index_select(0, idx))
    ks = raw(inp.kv_scales.index_select(1, idx)) if inp.kv_scales is not None else None
    maxb = max(1, max(nblk) if nblk else 1)
    table = np.full((len(seqs), maxb), -1, dtype=np.int32)
    for i, (b, n) in enumerate(zip(seqs, nblk)):
        table[i, :n] = [remap[int(p)] for p in lay.block_table[b, :n]]
    q = raw(inp.q[torch.tensor(seqs, device=inp.device, dtype=torch.long)])
    return oracle.paged_decode_attention(
        q=q, k_cache=kc, v_cache=vc, block_table=table,
        seq_lens=lay.seq_lens[seqs], softmax_scale=inp.softmax_scale,
        q_dtype=w.q_dtype, kv_dtype=w.kv_dtype, kv_scales=ks)


def errors(got: np.ndarray, ref: np.ndarray):
    diff = got - ref
    max_abs = float(np.max(np.abs(diff))) if diff.size else 0.0
    nref = float(np.linalg.norm(ref))
    rel_l2 = float(np.linalg.norm(diff) / nref) if nref > 0 else float(np.linalg.norm(diff))
    return max_abs, rel_l2


def assert_close(got: np.ndarray, ref: np.ndarray, kv_dtype: str, what="", bf16_out_rounding=False):
    """Whole-tensor max-abs and relative-L2 bounds per KV dtype.

    bf16_out_rounding adds the rounding of a bf16 output to the max-abs bound
    elementwise: round-to-nearest-even to bf16 (8 significant bits) moves a
    value by at most 2^-8 of its magnitude, which exceeds 1e-2 once |out| > 2.56
    (outputs that large occur only when a few tokens dominate the softmax).
    """
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    max_abs, rel_l2 = errors(got, ref)
    tol_abs, tol_rel = TOL[kv_dtype]
    if bf16_out_rounding:
        excess = np.abs(got - ref) - (tol_abs + 2.0 ** -8 * np.abs(ref))
        assert excess.max() <= 0, f"{what}: error exceeds 1e-2 + 2^-8|ref| by {excess.max():.3e}"
    else:
        assert max_abs <= tol_abs, f"{what}: max_abs {max_abs:.3e} > {tol_abs:.0e} (rel_l2 {rel_l2:.3e})"
    if tol_rel is not None:
        assert rel_l2 <= tol_rel, f"{what}: rel_l2 {rel_l2:.3e} > {tol_rel:.0e} (max_abs {max_abs:.3e})"
    return max_abs, rel_l2
