"""The stream-K partition's invariants, on a line-for-line Python model of the
two places that compute it: the decode driver's chunk walk (which blocks of
which (entry, KV head) unit each chunk runs) and the combine kernel's segment
count (which chunks hold a unit's partials). Exercised over random lengths,
KV heads, unit start costs and chunk sizes, including chunks shorter than a
start cost, which end inside it and hold none of that unit's blocks.

Invariants: every block of every unit is run by exactly one chunk, the
chunks of a unit run its blocks in order, and the combine's chunk list for a
unit is exactly the list of chunks that ran some of its blocks, so it never
merges a slot that was not written this call (and a unit run by a single
chunk is the one whose output that chunk writes directly)."""

import bisect
import math

import numpy as np
import pytest


def chunk_walk(nbs, hkv, f_cost, q):
    """The decode driver: chunk c covers stream units [c*q, (c+1)*q); an
    entry with nb > 0 blocks spans hkv units of f_cost + nb stream units, block
    j of KV head kvh starting at f_cost + j within its unit."""
    n_e = [nb + f_cost if nb > 0 else 0 for nb in nbs]
    cum = [0]
    for n in n_e:
        cum.append(cum[-1] + n)
    total = cum[-1] * hkv
    nchunks = (total + q - 1) // q if total else 0
    heads = [c * hkv for c in cum[:-1]]
    segs = {}
    for c in range(nchunks):
        pos, end = c * q, min(c * q + q, total)
        v = bisect.bisect_right(heads, pos) - 1  # last entry whose first unit is <= pos
        while pos < end and v < len(nbs):
            nb = nbs[v]
            f = f_cost if nb > 0 else 0
            nbw = f + nb
            base = cum[v] * hkv
            if pos >= base + nbw * hkv:
                v += 1
                continue
            rel = pos - base
            kvh = rel // nbw
            r0 = rel - kvh * nbw
            u0 = pos - r0
            r_end = min(end - u0, nbw)
            j_lo = r0 - f if r0 > f else 0
            j_hi = r_end - f if r_end > f else 0
            if j_lo < j_hi:
                segs.setdefault((v, kvh), []).append((c, j_lo, j_hi))
            pos = u0 + (f + j_hi if j_hi < nb else nbw)
    return cum, segs, nchunks


def combine_chunks(cum, v, kvh, nb, hkv, f_cost, q):
    """The combine kernel: from the chunk holding the unit's first block to
    the one holding its last."""
    start = cum[v] * hkv + kvh * (f_cost + nb) + f_cost
    w0 = start // q
    nseg = (start + nb - 1) // q - w0 + 1
    return list(range(w0, w0 + nseg))


def check(nbs, hkv, f_cost, q):
    cum, segs, nchunks = chunk_walk(nbs, hkv, f_cost, q)
    for v, nb in enumerate(nbs):
        for kvh in range(hkv):
            got = segs.get((v, kvh), [])
            if nb == 0:
                assert got == [], (v, kvh)
                continue
            # blocks 0 .. nb - 1 once each, in chunk order
            covered = [j for _, lo, hi in got for j in range(lo, hi)]
            assert covered == list(range(nb)), (nbs, hkv, f_cost, q, v, kvh, got)
            chunks = [c for c, _, _ in got]
            assert chunks == sorted(set(chunks))
            assert chunks == combine_chunks(cum, v, kvh, nb, hkv, f_cost, q), (nbs, hkv, f_cost, q, v, kvh)
            assert all(c < nchunks for c in chunks)


@pytest.mark.parametrize("seed", range(40))
def test_partition_random(seed):
    rng = np.random.default_rng(seed)
    E = int(rng.integers(1, 40))
    nbs = [int(x) if rng.random() > 0.2 else 0 for x in rng.integers(1, 120, E)]
    hkv = int(rng.integers(1, 9))
    f_cost = int(rng.choice([0, 1, 2, 4, 7]))
    total = sum(n + f_cost for n in nbs if n > 0) * hkv
    if total == 0:
        return
    for waves in (1, 3, 64, 1024):
        for min_share in (1, 8):
            q = max(math.ceil(total / waves), min_share)
            check(nbs, hkv, f_cost, q)
    for q in (1, 2, 3, 5):  # chunks shorter than a start cost
        check(nbs, hkv, f_cost, q)


def test_partition_edges():
    check([1], 1, 0, 1)
    check([1], 1, 4, 1)            # every chunk but the last is inside the start cost
    check([0, 0, 5, 0], 3, 2, 2)   # empty entries cost nothing
    check([16, 1, 16], 2, 4, 5)    # one-block units between longer ones
    check([100], 8, 2, 1000)       # one chunk holds everything: direct output
