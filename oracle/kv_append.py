"""Reference for appending one decode step's new keys and values to a paged
KV cache, including the fp8 (OCP E4M3) tile-scale policy.

TEST INFRASTRUCTURE ONLY (see the package docstring): never imported by the
product path.

Every decode step of the rollout phase (the paper's Sec. 2.2) produces one
new token per live sequence; before attention reads the cache, that token's
key and value are written into the sequence's paged cache (vLLM's paged KV
cache, which the paper cites in Sec. 8). The paper specifies no format; the
reading here is the library's: same layouts as ``decode_attention`` (K tile
[BS, D] token-major, V tile [D, BS] dim-major), and for fp8 caches one scale per
(block, KV head) tile and per K / V, kept at

    scale = max(amax / 448, 2^-126)

over the tokens written to the tile so far, so that a full tile ends with the
scale of the per-tile amax recipe (the fp8 workload's codes are produced that
way). When a new token's amax exceeds 448 * scale, the scale grows to the new
token's amax / 448 and the tile's earlier codes are re-encoded with it (their
decoded values times old / new scale); otherwise the scale stays and only the
new token is encoded. A tile's first token (slot 0) always sets a fresh scale.

Where floating point decides an integer code, the arithmetic is float32 with
one rounding per operation (IEEE multiply and correctly rounded divide), the
precision the kernel computes in, step for step:

    amax       = max_d |x_d|                         (exact)
    keep       = slot > 0 and old > 0 and amax <= fl(448 * old)
    new scale  = max(fl(amax / 448), 2^-126)         unless keep
    re-encode  = enc(fl(fl(dec(c) * old) / scale))   for earlier codes c
    new codes  = enc(fl(x_d / scale))

with enc the round-to-nearest-even encoding into E4M3 after clamping to
[-448, 448] (NaN stays NaN).
"""

import numpy as np

from .decode_attention import bf16_to_f64, e4m3fn_to_f64

E4M3_MAX = 448.0
MIN_SCALE = np.float32(2.0 ** -126)

# The 127 non-negative finite E4M3 values, by code 0x00 .. 0x7E (increasing).
_POS_CODES = np.arange(0x7F, dtype=np.uint8)
_POS_VALUES = e4m3fn_to_f64(_POS_CODES)


def encode_e4m3fn(z):
    """float32 values -> OCP E4M3 (fn) codes, round to nearest, ties to even.

    Written out from the definition: clamp to the largest finite magnitude
    (448), find the two representable neighbours of |z| among the 127
    non-negative finite values, take the nearer, and on a tie the one whose
    code (mantissa) is even; the sign bit is copied. NaN maps to 0x7F (S = 0)
    or 0xFF.
    """
    z = np.asarray(z, dtype=np.float32)
    v = z.astype(np.float64)
    sign = np.where(np.signbit(v), 0x80, 0).astype(np.uint8)
    a = np.minimum(np.abs(np.nan_to_num(v, nan=0.0)), E4M3_MAX)
    hi = np.searchsorted(_POS_VALUES, a, side="left")          # first value >= a
    lo = np.maximum(hi - 1, 0)
    d_lo = a - _POS_VALUES[lo]
    d_hi = _POS_VALUES[hi] - a
    pick_lo = (d_lo < d_hi) | ((d_lo == d_hi) & (lo % 2 == 0))
    code = np.where(_POS_VALUES[hi] == a, hi, np.where(pick_lo, lo, hi)).astype(np.uint8)
    return np.where(np.isnan(v), np.uint8(0x7F) | sign, code | sign).astype(np.uint8)


def encode_bf16(x):
    """float32 -> bfloat16 bit patterns, round to nearest, ties to even.

    The two candidates are the bfloat16 values next to x (the pattern with the
    low 16 bits dropped, and the next one away from zero); the nearer one wins,
    a tie goes to the even pattern. NaN stays a quiet NaN.
    """
    x = np.asarray(x, dtype=np.float32)
    bits = x.view(np.uint32).astype(np.uint64)
    down = bits >> 16
    up = down + 1
    vd = bf16_to_f64(down.astype(np.uint16))
    vu = bf16_to_f64((up & 0xFFFF).astype(np.uint16))
    exact = x.astype(np.float64)
    dd, du = np.abs(exact - vd), np.abs(vu - exact)
    take_down = (vd == exact) | (dd < du) | ((dd == du) & (down % 2 == 0))
    out = np.where(take_down, down, up).astype(np.uint16)
    return np.where(np.isnan(x), ((bits >> 16) | 0x40).astype(np.uint16), out).astype(np.uint16)


def _as_f32(x, dtype):
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32)
    if dtype == "bf16":
        return bf16_to_f64(x).astype(np.float32)
    raise ValueError(f"new keys / values must be f32 or bf16, not {dtype!r}")


def append_tile_fp8(codes, old_scale, slot, x):
    """One fp8 tile, viewed token-major as codes[BS, D] (uint8), receives token
    ``slot`` with float32 values x[D]. Returns (codes, scale) after the append."""
    codes = codes.copy()
    x = np.asarray(x, dtype=np.float32)
    amax = np.float32(np.max(np.abs(x)))
    old = np.float32(old_scale)
    keep = slot > 0 and old > 0 and amax <= np.float32(np.float32(E4M3_MAX) * old)
    if keep:
        scale = old
    else:
        scale = max(np.float32(amax / np.float32(E4M3_MAX)), MIN_SCALE)
        if slot > 0:
            prev = e4m3fn_to_f64(codes[:slot]).astype(np.float32)
            codes[:slot] = encode_e4m3fn((prev * old) / scale)
    codes[slot] = encode_e4m3fn(x / scale)
    return codes, scale


def paged_kv_append(k_new, v_new, k_cache, v_cache, kv_scales, block_table, positions, new_dtype, kv_dtype):
    """Write token positions[b] of every sequence b into the paged cache, in place.

    k_new, v_new   [B, Hkv, D]   new keys / values (f32, or bf16 bit patterns)
    k_cache        [NB, Hkv, BS, D], v_cache [NB, Hkv, D, BS]   (f32 / bf16 bits / fp8 codes)
    kv_scales      [2, NB, Hkv] float32 (fp8 only; index 0 = K, 1 = V)
    block_table    [B, max_blocks] int32, positions [B] int32

    A sequence with a negative position is skipped; a position at or past
    BS * max_blocks, or a block-table entry outside [0, NB), is skipped and
    reported. Returns the status bits (1: position past the table, 2: bad
    block id).
    """
    B, hkv, D = k_new.shape
    NB, _, BS, _ = k_cache.shape
    max_blocks = block_table.shape[1]
    status = 0
    for b in range(B):
        t = int(positions[b])
        if t < 0:
            continue
        if t >= BS * max_blocks:
            status |= 1
            continue
        p = int(block_table[b, t // BS])
        if not 0 <= p < NB:
            status |= 2
            continue
        o = t % BS
        for h in range(hkv):
            xk = _as_f32(k_new[b, h], new_dtype)
            xv = _as_f32(v_new[b, h], new_dtype)
            if kv_dtype == "f32":
                k_cache[p, h, o, :] = xk
                v_cache[p, h, :, o] = xv
            elif kv_dtype == "bf16":
                k_cache[p, h, o, :] = encode_bf16(xk)
                v_cache[p, h, :, o] = encode_bf16(xv)
            elif kv_dtype == "fp8_e4m3":
                codes, s = append_tile_fp8(k_cache[p, h], kv_scales[0, p, h], o, xk)
                k_cache[p, h] = codes
                kv_scales[0, p, h] = s
                codes, s = append_tile_fp8(v_cache[p, h].T, kv_scales[1, p, h], o, xv)
                v_cache[p, h] = codes.T
                kv_scales[1, p, h] = s
            else:
                raise ValueError(f"unknown cache dtype {kv_dtype!r}")
    return status
