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


def _sequence_job(inp, q, b, kind):
    """Sequence b of ``inp`` as a self-contained one-sequence oracle problem:
    its query rows, host copies of its own blocks, its block-table row
    renumbered to them (data movement only)."""
    w = inp.workload
    lay = inp.layout
    n = (int(lay.seq_lens[b]) + 15) // 16
    phys, local = np.unique(lay.block_table[b, :n].astype(np.int64), return_inverse=True)
    if phys.size == 0:
        phys, local = np.zeros(1, dtype=np.int64), np.zeros(0, dtype=np.int64)
    idx = torch.from_numpy(phys).to(inp.device)
    table = np.full((1, max(n, 1)), -1, dtype=np.int32)
    table[0, :n] = local
    kw = dict(q=raw(q[b:b + 1]), k_cache=raw(inp.k_cache.index_select(0, idx)),
              v_cache=raw(inp.v_cache.index_select(0, idx)), block_table=table,
              seq_lens=lay.seq_lens[b:b + 1].copy(), softmax_scale=inp.softmax_scale,
              q_dtype=w.q_dtype, kv_dtype=w.kv_dtype,
              kv_scales=raw(inp.kv_scales.index_select(1, idx)) if inp.kv_scales is not None else None)
    return kind, b, kw


def oracle_whole(inp, what="", q=None):
    """Oracle output for every sequence of ``inp`` ([B, Hq, D], or [B, Q, Hq, D]
    with several query tokens; ``q`` replaces inp.q), computed one sequence per
    job in the worker pool of ``tests._oracle_pool``; longest sequences first,
    so that the last jobs are short."""
    from tests import _oracle_pool as P

    q = inp.q if q is None else q
    lens = inp.layout.seq_lens
    B = len(lens)
    kind = "decode" if q.dim() == 3 else "multi_token"
    ref = np.zeros(tuple(q.shape), dtype=np.float64)

    def put(b, out):
        ref[b] = out[0]

    order = np.argsort(-lens.astype(np.int64), kind="stable")
    t = P.run_jobs((_sequence_job(inp, q, int(b), kind) for b in order), put,
                   progress=lambda done, s: print(f"[oracle] {what}: {done}/{B} sequences, {s:.0f} s", flush=True))
    print(f"[oracle] {what}: all {B} sequences ({int(lens.sum())} tokens) in {t:.1f} s on "
          f"{P.cores_used()} worker processes", flush=True)
    return ref


def _prefill_rows_job(pin, b, i0, i1):
    """Query rows i0 .. i1 - 1 of prefill sequence b as a self-contained oracle
    problem (data movement only). Row i sits at position L - n + i, so these
    rows are the last i1 - i0 query tokens of the same sequence cut to
    L - n + i1 tokens: its first blocks, copied out, with a block table
    renumbered to them."""
    c = pin.cache
    lay = c.layout
    n, L = int(pin.counts[b]), int(lay.seq_lens[b])
    Lc = L - n + i1
    nb = (max(Lc, 0) + 15) // 16
    phys, local = np.unique(lay.block_table[b, :nb].astype(np.int64), return_inverse=True)
    if phys.size == 0:
        phys, local = np.zeros(1, dtype=np.int64), np.zeros(0, dtype=np.int64)
    idx = torch.from_numpy(phys).to(c.k_cache.device)
    table = np.full((1, max(nb, 1)), -1, dtype=np.int32)
    table[0, :nb] = local
    r0 = int(pin.offsets[b])
    kw = dict(q=raw(pin.q[r0 + i0:r0 + i1]), q_offsets=np.array([0, i1 - i0], dtype=np.int32),
              k_cache=raw(c.k_cache.index_select(0, idx)), v_cache=raw(c.v_cache.index_select(0, idx)),
              block_table=table, seq_lens=np.array([max(Lc, 0)], dtype=np.int32), softmax_scale=c.softmax_scale,
              q_dtype="bf16", kv_dtype=c.workload.kv_dtype,
              kv_scales=raw(c.kv_scales.index_select(1, idx)) if c.kv_scales is not None else None)
    return "prefill", (r0 + i0, r0 + i1), kw


def oracle_prefill_whole(pin, what="", rows_per_job=64):
    """Oracle output [T, Hq, D] of every query row of prefill ``pin``, computed
    over slices of ``rows_per_job`` rows in the worker pool of
    ``tests._oracle_pool``, longest sequences first."""
    from tests import _oracle_pool as P

    T = int(pin.q.shape[0])
    ref = np.zeros(tuple(pin.q.shape), dtype=np.float64)

    def put(rows, out):
        ref[rows[0]:rows[1]] = out

    lens = pin.cache.layout.seq_lens
    slices = ((int(b), i0, min(i0 + rows_per_job, int(pin.counts[b])))
              for b in np.argsort(-lens.astype(np.int64), kind="stable")
              for i0 in range(0, int(pin.counts[b]), rows_per_job))
    t = P.run_jobs((_prefill_rows_job(pin, b, i0, i1) for b, i0, i1 in slices), put,
                   progress=lambda done, s: print(f"[oracle] {what}: {done} row slices, {s:.0f} s", flush=True))
    print(f"[oracle] {what}: {T} rows in {t:.1f} s on {P.cores_used()} worker processes", flush=True)
    return ref


def worst_row_rel_l2(got: np.ndarray, ref: np.ndarray):
    """Largest relative L2 error of one output row (one sequence and query
    head, over D), with its index; rows whose reference is zero use the
    absolute norm. A diagnostic beside the whole-tensor bounds."""
    d = got.shape[-1]
    g = got.reshape(-1, d)
    r = ref.reshape(-1, d)
    num = np.linalg.norm(g - r, axis=1)
    den = np.linalg.norm(r, axis=1)
    rel = np.where(den > 0, num / np.where(den > 0, den, 1.0), num)
    i = int(np.argmax(rel))
    return float(rel[i]), np.unravel_index(i, got.shape[:-1])


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
