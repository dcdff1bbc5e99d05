"""GPU parity of the paged KV append (pda_paged_kv_append) against the oracle
(oracle/kv_append.py): caches and fp8 scales must match bit for bit, since the
append only moves and encodes values (every code decision is float32 on both
sides, with correctly rounded division)."""

import numpy as np
import pytest
import torch

import oracle

from tests import _gpu_util as U

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TORCH = {"f32": torch.float32, "bf16": torch.bfloat16}


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    from paper_2605_20863_amd import _lib
    return _lib


def make_cache(kv, NB, hkv, d, rng):
    """Host cache (raw stored patterns) and scales with arbitrary prior contents."""
    if kv == "f32":
        k = rng.standard_normal((NB, hkv, 16, d)).astype(np.float32)
        v = rng.standard_normal((NB, hkv, d, 16)).astype(np.float32)
    elif kv == "bf16":
        k = U.raw(torch.from_numpy(rng.standard_normal((NB, hkv, 16, d)).astype(np.float32)).to(torch.bfloat16))
        v = U.raw(torch.from_numpy(rng.standard_normal((NB, hkv, d, 16)).astype(np.float32)).to(torch.bfloat16))
    else:
        k = rng.integers(0, 0x7E, (NB, hkv, 16, d)).astype(np.uint8)
        v = rng.integers(0, 0x7E, (NB, hkv, d, 16)).astype(np.uint8)
    scales = rng.uniform(0.002, 0.02, (2, NB, hkv)).astype(np.float32)
    return k, v, scales


def to_dev(arr, kv):
    t = torch.from_numpy(np.ascontiguousarray(arr))
    if kv == "bf16":
        t = t.view(torch.bfloat16)
    return t.to(DEV)


def gpu_append(lib, kn, vn, k, v, scales, table, positions, kv):
    kc, vc = to_dev(k, kv), to_dev(v, kv)
    sc = torch.from_numpy(scales.copy()).to(DEV) if kv == "fp8_e4m3" else None
    lib.paged_kv_append(kn, vn, kc, vc, sc, torch.from_numpy(table).to(DEV), torch.from_numpy(positions).to(DEV))
    torch.cuda.synchronize()
    return U.raw(kc), U.raw(vc), (sc.cpu().numpy() if sc is not None else None)


def new_values(rng, B, hkv, d, new_dtype, amp=None):
    amp = np.ones((B, hkv, 1)) if amp is None else amp
    kn = torch.from_numpy((rng.standard_normal((B, hkv, d)) * amp).astype(np.float32)).to(TORCH[new_dtype])
    vn = torch.from_numpy((rng.standard_normal((B, hkv, d)) * amp).astype(np.float32)).to(TORCH[new_dtype])
    return kn.to(DEV), vn.to(DEV)


def check(lib, kn, vn, k, v, scales, table, positions, kv, new_dtype, what):
    gk, gv, gs = gpu_append(lib, kn, vn, k, v, scales, table, positions, kv)
    ok, ov, os_ = k.copy(), v.copy(), scales.copy()
    st = oracle.paged_kv_append(U.raw(kn), U.raw(vn), ok, ov, os_, table, positions, new_dtype, kv)
    assert np.array_equal(gk, ok), f"{what}: K cache differs at {np.argwhere(gk != ok)[:5].tolist()}"
    assert np.array_equal(gv, ov), f"{what}: V cache differs at {np.argwhere(gv != ov)[:5].tolist()}"
    if kv == "fp8_e4m3":
        assert np.array_equal(gs, os_), f"{what}: scales differ"
    assert lib.read_device_status() == st
    return ok, ov, os_


@pytest.mark.parametrize("kv", ["f32", "bf16", "fp8_e4m3"])
@pytest.mark.parametrize("new_dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [64, 128])
def test_append_matches_oracle(lib, kv, new_dtype, d):
    rng = np.random.default_rng(hash((kv, new_dtype, d)) % 2 ** 32)
    B, hkv, NB, maxb = 37, 4, 200, 5
    table = rng.permutation(NB)[:B * maxb].reshape(B, maxb).astype(np.int32)   # private blocks
    positions = rng.integers(0, 16 * maxb, B).astype(np.int32)
    positions[:6] = [0, 15, 16, 31, 79, 40]          # first and last slots of blocks
    k, v, scales = make_cache(kv, NB, hkv, d, rng)
    # token amplitudes that sometimes keep, sometimes grow the tile scale
    amp = rng.choice([0.01, 0.5, 3.0, 40.0], (B, hkv, 1))
    kn, vn = new_values(rng, B, hkv, d, new_dtype, amp)
    print(f"[append] kv={kv} new={new_dtype} D={d}", flush=True)
    check(lib, kn, vn, k, v, scales, table, positions, kv, new_dtype, f"{kv}/{new_dtype}/D{d}")


def test_append_encoding_ties_and_subnormals(lib):
    """Slot 0 of fresh tiles with one element at 448 sets the scale to exactly 1,
    so the other elements encode as themselves: ties (to even), subnormals,
    signed zeros and the largest values go through the kernel's conversion."""
    vals = oracle.e4m3fn_to_f64(np.arange(0x7F, dtype=np.uint8))
    mids = ((vals[1:] + vals[:-1]) / 2).astype(np.float32)
    z = np.concatenate([vals.astype(np.float32), mids, np.nextafter(mids, np.float32(0)),
                        np.nextafter(mids, np.float32(1000)), [0.0, -0.0, 2.0 ** -10, 447.9, 440.0]]).astype(np.float32)
    z = np.concatenate([z, -z])
    d, hkv = 128, 1
    per = d - 1
    B = -(-len(z) // per)
    z = np.concatenate([z, np.zeros(B * per - len(z), np.float32)]).reshape(B, per)
    x = np.concatenate([np.full((B, 1), 448.0, np.float32), z], axis=1)[:, None, :]
    NB = B + 3
    table = np.arange(B, dtype=np.int32)[:, None]
    positions = np.zeros(B, np.int32)
    rng = np.random.default_rng(3)
    k, v, scales = make_cache("fp8_e4m3", NB, hkv, d, rng)
    kn = torch.from_numpy(x).to(DEV)
    vn = torch.from_numpy(-x).to(DEV)
    _, _, s = check(lib, kn, vn, k, v, scales, table, positions, "fp8_e4m3", "f32", "ties")
    assert (s[:, :B] == 1.0).all()


def test_append_many_steps_fp8(lib):
    """48 decode steps into empty fp8 tiles with token scales varying over three
    decades: scales grow, earlier codes are re-encoded, and cache and scales stay
    identical to the oracle's after every step."""
    rng = np.random.default_rng(21)
    B, hkv, d, NB, maxb = 6, 2, 128, 40, 4
    table = rng.permutation(NB)[:B * maxb].reshape(B, maxb).astype(np.int32)
    k, v, scales = make_cache("fp8_e4m3", NB, hkv, d, rng)
    gk, gv, gs = to_dev(k, "fp8_e4m3"), to_dev(v, "fp8_e4m3"), torch.from_numpy(scales.copy()).to(DEV)
    tdev = torch.from_numpy(table).to(DEV)
    for step in range(48):
        positions = np.full(B, step, np.int32)
        positions[0] = -1 if step % 7 == 3 else step      # a sequence that sits out some steps
        amp = np.exp(rng.uniform(-3, 3, (B, hkv, 1)))
        kn, vn = new_values(rng, B, hkv, d, "bf16", amp)
        lib.paged_kv_append(kn, vn, gk, gv, gs, tdev, torch.from_numpy(positions).to(DEV))
        oracle.paged_kv_append(U.raw(kn), U.raw(vn), k, v, scales, table, positions, "bf16", "fp8_e4m3")
    torch.cuda.synchronize()
    assert np.array_equal(U.raw(gk), k) and np.array_equal(U.raw(gv), v)
    assert np.array_equal(gs.cpu().numpy(), scales)
    assert lib.read_device_status() == 0


def test_append_skips_and_flags(lib):
    rng = np.random.default_rng(31)
    B, hkv, d, NB = 5, 2, 64, 12
    table = np.array([[4, 1, -1], [2, 5, 0], [3, 3, 3], [99, 9, 9], [0, 1, 2]], dtype=np.int32)
    positions = np.array([17, 5, -1, 0, 48], dtype=np.int32)   # seq 2 skipped, 3: bad id, 4: past the table
    for kv in ("bf16", "fp8_e4m3"):
        k, v, scales = make_cache(kv, NB, hkv, d, rng)
        kn, vn = new_values(rng, B, hkv, d, "f32")
        check(lib, kn, vn, k, v, scales, table, positions, kv, "f32", f"flags {kv}")


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_append_then_decode(lib, kv):
    """Sequences built token by token with the append kernel, then attended by
    the decode kernel, against the oracle's append and attention."""
    rng = np.random.default_rng(41)
    B, hkv, G, d, maxb = 6, 2, 4, 128, 6
    NB = B * maxb + 4
    lens = rng.integers(1, 16 * maxb, B).astype(np.int32)
    table = rng.permutation(NB)[:B * maxb].reshape(B, maxb).astype(np.int32)
    k, v, scales = make_cache(kv, NB, hkv, d, rng)
    gk, gv = to_dev(k, kv), to_dev(v, kv)
    gs = torch.from_numpy(scales.copy()).to(DEV) if kv == "fp8_e4m3" else None
    tdev = torch.from_numpy(table).to(DEV)
    for t in range(int(lens.max())):
        positions = np.where(t < lens, t, -1).astype(np.int32)
        kn, vn = new_values(rng, B, hkv, d, "bf16")
        lib.paged_kv_append(kn, vn, gk, gv, gs, tdev, torch.from_numpy(positions).to(DEV))
        oracle.paged_kv_append(U.raw(kn), U.raw(vn), k, v, scales, table, positions, "bf16", kv)
    q = torch.from_numpy(rng.standard_normal((B, hkv * G, d)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    out = torch.empty_like(q)
    lib.paged_decode_attention(q, gk, gv, tdev, torch.from_numpy(lens).to(DEV), gs, out, d ** -0.5)
    torch.cuda.synchronize()
    assert np.array_equal(U.raw(gk), k) and np.array_equal(U.raw(gv), v)
    ref = oracle.paged_decode_attention(q=U.raw(q), k_cache=k, v_cache=v, block_table=table, seq_lens=lens,
                                        softmax_scale=d ** -0.5, q_dtype="bf16", kv_dtype=kv,
                                        kv_scales=scales if kv == "fp8_e4m3" else None)
    U.assert_close(U.out_to_f64(out), ref, kv, f"append then decode {kv}")
    assert lib.read_device_status() == 0
