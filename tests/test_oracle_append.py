"""Pins of the KV-append oracle (oracle/kv_append.py) to things other than itself.

* The E4M3 and bfloat16 encoders: exhaustive round trips, hand-derived ties,
  saturation and NaN, and agreement with torch's independent float8_e4m3fn /
  bfloat16 conversions.
* The fp8 tile-scale policy: closed forms for a fresh tile, the per-tile amax
  recipe (written here with torch) when the largest token comes first, exact
  re-encoding when the scale doubles, an unchanged tile when the scale holds.
* Placement: K rows and dim-major V columns land where the decode oracle reads
  them, nothing else changes, skipped / reported positions and block ids, and
  appending a sequence token by token reproduces attention over its raw keys.

``test_append_mutants_are_caught`` plants plausible mistakes in the oracle and
checks that at least one pin fails for each.
"""

import numpy as np
import pytest
import torch

import oracle
import oracle.kv_append as ka


def _torch_e4m3(z):
    return torch.from_numpy(np.asarray(z, dtype=np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def _torch_bf16(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def pin_e4m3_roundtrip(o):
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    vals = oracle.e4m3fn_to_f64(codes).astype(np.float32)
    assert np.array_equal(o.encode_e4m3fn(vals), codes)


def pin_e4m3_hand_ties(o):
    cases = [(1.0625, 0x38), (1.1875, 0x3A), (2.0 ** -10, 0x00), (1.5 * 2.0 ** -9, 0x02), (-1.0625, 0xB8),
             (448.0, 0x7E), (464.0, 0x7E), (1e6, 0x7E), (-1e6, 0xFE), (0.0, 0x00), (-0.0, 0x80),
             (2.0 ** -6, 0x08), (240.0, 0x77), (0.8125, 0x35)]
    z = np.array([c[0] for c in cases], dtype=np.float32)
    assert np.array_equal(o.encode_e4m3fn(z), np.array([c[1] for c in cases], dtype=np.uint8))
    assert o.encode_e4m3fn(np.array([np.nan], dtype=np.float32))[0] & 0x7F == 0x7F


def pin_e4m3_vs_torch(o):
    vals = oracle.e4m3fn_to_f64(np.arange(0x7F, dtype=np.uint8))
    mids = (vals[1:] + vals[:-1]) / 2
    z = np.concatenate([vals, mids, np.nextafter(mids.astype(np.float32), 0), np.nextafter(mids.astype(np.float32), 1000)])
    z = np.concatenate([z, -z, np.random.default_rng(7).uniform(-448, 448, 4000)]).astype(np.float32)
    assert np.array_equal(o.encode_e4m3fn(z), _torch_e4m3(z))


def pin_bf16(o):
    x = np.concatenate([np.random.default_rng(8).standard_normal(3000) * 10,
                        [1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(1 + 2.0 ** -8), 3.0, 0.0, 1e-40]]).astype(np.float32)
    assert np.array_equal(o.encode_bf16(x), _torch_bf16(x))
    assert o.encode_bf16(np.float32([1 + 2.0 ** -8]))[0] == 0x3F80          # tie -> even
    assert o.encode_bf16(np.float32([1 + 3 * 2.0 ** -8]))[0] == 0x3F82


def pin_fresh_tile(o):
    rng = np.random.default_rng(9)
    x = rng.standard_normal(64).astype(np.float32)
    stale = np.full((16, 64), 0x33, dtype=np.uint8)
    codes, s = o.append_tile_fp8(stale, np.float32(1e-3), 0, x)   # a stale scale is ignored at slot 0
    amax = np.float32(np.abs(x).max())
    assert s == np.float32(amax / np.float32(448))
    i = int(np.argmax(np.abs(x)))
    assert codes[0, i] == (0x7E if x[i] > 0 else 0xFE)
    assert np.array_equal(codes[1:], stale[1:])
    # an all-zero token: the scale floor keeps codes finite
    codes, s = o.append_tile_fp8(stale, np.float32(0), 0, np.zeros(64, np.float32))
    assert s == np.float32(2.0 ** -126) and not codes[0].any()


def pin_tile_recipe(o):
    """Largest token first: the scale never moves and the tile equals the
    per-tile recipe (amax / 448 over the tile, clamp, round to E4M3)."""
    rng = np.random.default_rng(10)
    x = rng.standard_normal((16, 128)).astype(np.float32)
    order = np.argsort(-np.abs(x).max(axis=1))
    x = x[order]
    codes = np.zeros((16, 128), np.uint8)
    s = np.float32(0)
    for t in range(16):
        codes, s = o.append_tile_fp8(codes, s, t, x[t])
    xt = torch.from_numpy(x)
    scale = torch.clamp(xt.abs().amax() / 448.0, min=2.0 ** -126)
    ref = torch.clamp(xt / scale, -448, 448).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert s == np.float32(scale.item())
    assert np.array_equal(codes, ref)


def pin_scale_growth(o):
    """A token with twice the amax doubles the scale; earlier values, re-encoded,
    decode to exactly the same reals (halving a normal E4M3 value is exact)."""
    rng = np.random.default_rng(11)
    x0 = rng.uniform(0.25, 1.0, 64).astype(np.float32) * rng.choice([-1, 1], 64).astype(np.float32)
    x0[0] = 1.0
    codes, s0 = o.append_tile_fp8(np.zeros((16, 64), np.uint8), 0, 0, x0)
    before = oracle.e4m3fn_to_f64(codes[0]) * float(s0)
    x1 = np.zeros(64, np.float32)
    x1[3] = 2.0
    codes2, s1 = o.append_tile_fp8(codes, s0, 1, x1)
    assert s1 == np.float32(2 * s0)
    assert np.array_equal(oracle.e4m3fn_to_f64(codes2[0]) * float(s1), before)
    assert not np.array_equal(codes2[0], codes[0])
    # a smaller token keeps the scale and the earlier codes
    codes3, s2 = o.append_tile_fp8(codes2, s1, 2, x0 * np.float32(0.5))
    assert s2 == s1 and np.array_equal(codes3[:2], codes2[:2])


def pin_scale_growth_non_pow2(o):
    """A token whose amax is 1.37 times the tile's grows the scale by a factor
    that is not a power of two. The new scale is the token's amax / 448, and
    every re-encoded code is a nearest E4M3 neighbour of the exact real
    dec(c) * old / new (fp64 here), up to the float32 rounding of that
    quotient: a re-encode that truncates, or that drops the division by the
    new scale, is caught (a power-of-two growth cannot tell them apart)."""
    rng = np.random.default_rng(21)
    x0 = rng.standard_normal((3, 64)).astype(np.float32)
    codes, s = np.zeros((16, 64), np.uint8), np.float32(0)
    for t in range(3):
        codes, s = o.append_tile_fp8(codes, s, t, x0[t])
    amax0 = np.float32(np.abs(x0).max())
    assert s == np.float32(amax0 / np.float32(448))   # the largest of the first tokens set it
    x1 = rng.standard_normal(64).astype(np.float32)
    x1 = (x1 * np.float32(1.37 * amax0 / np.abs(x1).max())).astype(np.float32)
    grown, s1 = o.append_tile_fp8(codes, s, 3, x1)
    assert s1 == np.float32(np.float32(np.abs(x1).max()) / np.float32(448))
    ratio = float(s) / float(s1)
    assert abs(np.log2(ratio) - np.rint(np.log2(ratio))) > 0.1, "growth must not be a power of two"
    z = (oracle.e4m3fn_to_f64(codes[:3]) * float(s) / float(s1)).ravel()
    got = oracle.e4m3fn_to_f64(grown[:3]).ravel()
    finite = oracle.e4m3fn_to_f64(np.array([c for c in range(256) if c & 0x7F != 0x7F], np.uint8))
    dmin = np.min(np.abs(finite[None, :] - z[:, None]), axis=1)
    assert np.all(np.abs(got - z) <= dmin + 2.0 ** -22 * np.abs(z))
    assert np.all((got == 0) | (np.sign(got) == np.sign(z)))
    assert not np.array_equal(grown[:3], codes[:3])
    assert np.array_equal(grown[4:], codes[4:])      # slots past the new token are untouched


def _cache(kv, NB=6, hkv=2, d=64, seed=12):
    rng = np.random.default_rng(seed)
    if kv == "f32":
        k = rng.standard_normal((NB, hkv, 16, d)).astype(np.float32)
        v = rng.standard_normal((NB, hkv, d, 16)).astype(np.float32)
    elif kv == "bf16":
        k = rng.integers(0, 0x3F00, (NB, hkv, 16, d)).astype(np.uint16)
        v = rng.integers(0, 0x3F00, (NB, hkv, d, 16)).astype(np.uint16)
    else:
        k = rng.integers(0, 0x70, (NB, hkv, 16, d)).astype(np.uint8)
        v = rng.integers(0, 0x70, (NB, hkv, d, 16)).astype(np.uint8)
    scales = rng.uniform(0.001, 0.01, (2, NB, hkv)).astype(np.float32)
    return k, v, scales


def pin_placement_and_flags(o):
    rng = np.random.default_rng(13)
    table = np.array([[4, 1, -1], [2, 5, 0], [3, 3, 3], [9, 9, 9], [0, 1, 2]], dtype=np.int32)
    positions = np.array([17, 5, -1, 0, 48], dtype=np.int32)   # seq 2 skipped, 3: bad id, 4: past the table
    for kv in ("f32", "bf16"):
        k, v, sc = _cache(kv)
        k0, v0 = k.copy(), v.copy()
        kn = rng.standard_normal((5, 2, 64)).astype(np.float32)
        vn = rng.standard_normal((5, 2, 64)).astype(np.float32)
        st = o.paged_kv_append(kn, vn, k, v, sc, table, positions, "f32", kv)
        assert st == 3
        enc = (lambda a: a) if kv == "f32" else o.encode_bf16
        ek, ev = k0.copy(), v0.copy()
        ek[1, :, 1, :] = enc(kn[0])        # token 17 of seq 0 -> block 1, slot 1
        ev[1, :, :, 1] = enc(vn[0])
        ek[2, :, 5, :] = enc(kn[1])        # token 5 of seq 1 -> block 2, slot 5
        ev[2, :, :, 5] = enc(vn[1])
        assert np.array_equal(k, ek) and np.array_equal(v, ev)


def pin_append_then_attend(o):
    """Appending a sequence token by token into an f32 cache, then attending,
    equals attention over the raw keys and values."""
    rng = np.random.default_rng(14)
    L, hkv, G, d = 37, 2, 3, 32
    K = rng.standard_normal((L, hkv, d)).astype(np.float32)
    V = rng.standard_normal((L, hkv, d)).astype(np.float32)
    kc = np.full((5, hkv, 16, d), np.nan, np.float32)
    vc = np.full((5, hkv, d, 16), np.nan, np.float32)
    table = np.array([[3, 0, 4]], dtype=np.int32)
    for t in range(L):
        assert o.paged_kv_append(K[None, t], V[None, t], kc, vc, None, table, np.array([t], np.int32),
                                 "f32", "f32") == 0
    q = rng.standard_normal((1, hkv * G, d)).astype(np.float32)
    out = oracle.paged_decode_attention(q=q, k_cache=kc, v_cache=vc, block_table=table,
                                        seq_lens=np.array([L], np.int32), softmax_scale=0.2, q_dtype="f32",
                                        kv_dtype="f32")
    for h in range(hkv * G):
        ref = oracle.attend(q[0, h].astype(np.float64), K[:, h // G].astype(np.float64),
                            V[:, h // G].astype(np.float64), 0.2)
        assert np.allclose(out[0, h], ref, rtol=0, atol=1e-12)


def pin_fp8_cache(o):
    """fp8 cache: the K tile row and the V tile column of the new token hold the
    codes of the tile policy, and the scales are stored per K / V."""
    rng = np.random.default_rng(15)
    k, v, sc = _cache("fp8_e4m3")
    table = np.array([[4, 1], [2, 5]], dtype=np.int32)
    positions = np.array([16 + 3, 0], dtype=np.int32)
    kn = rng.standard_normal((2, 2, 64)).astype(np.float32)
    vn = rng.standard_normal((2, 2, 64)).astype(np.float32)
    k0, v0, sc0 = k.copy(), v.copy(), sc.copy()
    assert o.paged_kv_append(kn, vn, k, v, sc, table, positions, "f32", "fp8_e4m3") == 0
    for h in range(2):
        ck, s = o.append_tile_fp8(k0[1, h], sc0[0, 1, h], 3, kn[0, h])
        assert np.array_equal(k[1, h], ck) and sc[0, 1, h] == s
        cv, s = o.append_tile_fp8(v0[1, h].T, sc0[1, 1, h], 3, vn[0, h])
        assert np.array_equal(v[1, h], cv.T) and sc[1, 1, h] == s
        assert sc[0, 2, h] == np.float32(np.float32(np.abs(kn[1, h]).max()) / np.float32(448))
    assert np.array_equal(k[[0, 3, 4, 5]], k0[[0, 3, 4, 5]])


PINS = [pin_e4m3_roundtrip, pin_e4m3_hand_ties, pin_e4m3_vs_torch, pin_bf16, pin_fresh_tile, pin_tile_recipe,
        pin_scale_growth, pin_scale_growth_non_pow2, pin_placement_and_flags, pin_append_then_attend, pin_fp8_cache]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_append_pin(pin):
    pin(ka)


# ----------------------------------------------------------------- planted mistakes

def _mut_ties_away(mp):
    orig = ka.encode_e4m3fn

    def bad(z):
        z = np.asarray(z, dtype=np.float32)
        out = orig(z)
        vals = oracle.e4m3fn_to_f64(out)
        up = orig(np.nextafter(z, np.where(z >= 0, np.float32(1e9), np.float32(-1e9)).astype(np.float32)))
        tie = np.abs(np.abs(z.astype(np.float64)) - np.abs(vals)) == np.abs(np.abs(oracle.e4m3fn_to_f64(up))
                                                                           - np.abs(z.astype(np.float64)))
        return np.where(tie & (up != out), up, out).astype(np.uint8)
    mp.setattr(ka, "encode_e4m3fn", bad)


def _mut_overflow_nan(mp):
    orig = ka.encode_e4m3fn
    mp.setattr(ka, "encode_e4m3fn",
               lambda z: np.where(np.abs(np.asarray(z, np.float32)) > 448, np.uint8(0x7F), orig(z)).astype(np.uint8))


def _mut_bf16_truncate(mp):
    mp.setattr(ka, "encode_bf16",
               lambda x: (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16))


def _mut_scale_never_grows(mp):
    orig = ka.append_tile_fp8

    def bad(codes, old, slot, x):
        if slot > 0 and old > 0:
            codes = codes.copy()
            codes[slot] = ka.encode_e4m3fn(np.asarray(x, np.float32) / np.float32(old))
            return codes, np.float32(old)
        return orig(codes, old, slot, x)
    mp.setattr(ka, "append_tile_fp8", bad)


def _mut_no_reencode(mp):
    orig = ka.append_tile_fp8

    def bad(codes, old, slot, x):
        new, s = orig(codes, old, slot, x)
        new[:slot] = codes[:slot]
        return new, s
    mp.setattr(ka, "append_tile_fp8", bad)


def _mut_slot0_keeps_scale(mp):
    orig = ka.append_tile_fp8

    def bad(codes, old, slot, x):
        if slot == 0 and old > 0:        # a reused block keeps its stale scale
            codes = codes.copy()
            codes[0] = ka.encode_e4m3fn(np.asarray(x, np.float32) / np.float32(old))
            return codes, np.float32(old)
        return orig(codes, old, slot, x)
    mp.setattr(ka, "append_tile_fp8", bad)


def _mut_v_token_major(mp):
    orig = ka.paged_kv_append

    def bad(k_new, v_new, k_cache, v_cache, kv_scales, block_table, positions, new_dtype, kv_dtype):
        vt = np.ascontiguousarray(np.swapaxes(v_cache, 2, 3))
        st = orig(k_new, v_new, k_cache, vt, kv_scales, block_table, positions, new_dtype, kv_dtype)
        v_cache[...] = vt.reshape(v_cache.shape)
        return st
    mp.setattr(ka, "paged_kv_append", bad)


def _reencode_variant(mp, reencode):
    """The oracle's tile policy with its re-encode step replaced."""
    def bad(codes, old_scale, slot, x):
        codes = codes.copy()
        x = np.asarray(x, dtype=np.float32)
        amax = np.float32(np.max(np.abs(x)))
        old = np.float32(old_scale)
        keep = slot > 0 and old > 0 and amax <= np.float32(np.float32(448) * old)
        if keep:
            scale = old
        else:
            scale = max(np.float32(amax / np.float32(448)), np.float32(2.0 ** -126))
            if slot > 0:
                codes[:slot] = reencode(oracle.e4m3fn_to_f64(codes[:slot]).astype(np.float32), old, scale)
        codes[slot] = ka.encode_e4m3fn(x / scale)
        return codes, scale
    mp.setattr(ka, "append_tile_fp8", bad)


def _mut_reencode_truncates(mp):
    vals = oracle.e4m3fn_to_f64(np.arange(0x7F, dtype=np.uint8))

    def trunc(prev, old, scale):  # round toward zero instead of to nearest
        z = np.minimum(np.abs((prev * old) / scale).astype(np.float64), 448.0)
        code = (np.searchsorted(vals, z, side="right") - 1).astype(np.uint8)
        return np.where(np.signbit((prev * old) / scale), code | 0x80, code).astype(np.uint8)
    _reencode_variant(mp, trunc)


def _mut_reencode_drops_division(mp):
    _reencode_variant(mp, lambda prev, old, scale: ka.encode_e4m3fn(prev * old))


MUTANTS = {
    "fp8_reencode_truncates": _mut_reencode_truncates,
    "fp8_reencode_drops_division": _mut_reencode_drops_division,
    "e4m3_ties_away_from_zero": _mut_ties_away,
    "e4m3_overflow_to_nan": _mut_overflow_nan,
    "bf16_truncated": _mut_bf16_truncate,
    "fp8_scale_never_grows": _mut_scale_never_grows,
    "fp8_no_reencode_on_growth": _mut_no_reencode,
    "fp8_slot0_keeps_stale_scale": _mut_slot0_keeps_scale,
    "v_written_token_major": _mut_v_token_major,
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_append_mutants_are_caught(name, monkeypatch):
    MUTANTS[name](monkeypatch)
    failed = []
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin(ka)
        except Exception:  # noqa: BLE001 - any failure counts as caught
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
