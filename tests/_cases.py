"""Small paged decode problems built independently of the oracle.

Each case starts from *contiguous* per-sequence keys and values whose float64
values are known exactly (decoded with torch, not with the oracle's decoders),
then scatters them into the documented paged layout with this module's own
indexing:

    k_cache [NB, Hkv, BS, D], v_cache [NB, Hkv, D, BS], kv_scales [2, NB, Hkv]

so a pin comparing the oracle on the paged arrays with an independent
computation on the contiguous arrays checks the oracle's gather, layout and
decoding as well as its arithmetic.
"""

import dataclasses

import numpy as np
import torch

BS = 16


@dataclasses.dataclass
class Case:
    q: np.ndarray            # stored q (float32 or uint16 bf16 bits)
    q64: np.ndarray          # [B, Hq, D] exact float64 values of q
    k_cache: np.ndarray
    v_cache: np.ndarray
    block_table: np.ndarray
    seq_lens: np.ndarray
    kv_scales: np.ndarray    # [2, NB, Hkv] (ones unless fp8)
    K64: list                # per b: [L_b, Hkv, D] exact float64 keys (scaled)
    V64: list                # per b: [L_b, Hkv, D] exact float64 values (scaled)
    q_dtype: str
    kv_dtype: str
    softmax_scale: float

    def oracle_args(self):
        return dict(q=self.q, k_cache=self.k_cache, v_cache=self.v_cache,
                    block_table=self.block_table, seq_lens=self.seq_lens,
                    softmax_scale=self.softmax_scale, q_dtype=self.q_dtype,
                    kv_dtype=self.kv_dtype,
                    kv_scales=self.kv_scales if self.kv_dtype == "fp8_e4m3" else None)


def _store(x, dtype):
    """float64 array -> (stored array, exact float64 of what is stored) via torch."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64))
    if dtype == "f32":
        s = t.to(torch.float32)
        return s.numpy(), s.to(torch.float64).numpy()
    if dtype == "bf16":
        s = t.to(torch.bfloat16)
        return s.view(torch.int16).numpy().view(np.uint16), s.to(torch.float64).numpy()
    if dtype == "fp8_e4m3":
        s = t.clamp(-448, 448).to(torch.float8_e4m3fn)
        return s.view(torch.uint8).numpy(), s.to(torch.float64).numpy()
    raise ValueError(dtype)


def nan_code(dtype):
    return {"f32": np.float32("nan"), "bf16": np.uint16(0x7FC0), "fp8_e4m3": np.uint8(0x7F)}[dtype]


def build(lens, hq, hkv, d, kv_dtype="f32", q_dtype=None, seed=0, softmax_scale=None,
          spare=3, poison=True, key_fn=None, value_fn=None, q_fn=None, perm=None,
          fp8_headroom=1.37):
    """Random paged problem with the given sequence lengths.

    key_fn / value_fn / q_fn, when given, replace the N(0,1) draws: they take
    (rng, shape) and return float64 arrays (before rounding to storage).
    """
    rng = np.random.default_rng(seed)
    q_dtype = q_dtype or ("f32" if kv_dtype == "f32" else "bf16")
    softmax_scale = 1.0 / np.sqrt(d) if softmax_scale is None else softmax_scale
    lens = np.asarray(lens, dtype=np.int32)
    B = len(lens)
    nblk = [(int(L) + BS - 1) // BS for L in lens]
    used = sum(nblk)
    NB = used + spare
    perm = rng.permutation(NB) if perm is None else np.asarray(perm)
    maxb = max(1, max(nblk) if nblk else 1)
    table = np.full((B, maxb), -1, dtype=np.int32)
    nxt = 0
    for b in range(B):
        for j in range(nblk[b]):
            table[b, j] = perm[nxt]
            nxt += 1

    draw = lambda fn, shape: (fn(rng, shape) if fn else rng.standard_normal(shape))
    qraw = draw(q_fn, (B, hq, d))
    q, q64 = _store(qraw, q_dtype)

    if kv_dtype == "fp8_e4m3":
        store_dt = np.uint8
    elif kv_dtype == "bf16":
        store_dt = np.uint16
    else:
        store_dt = np.float32
    k_cache = np.full((NB, hkv, BS, d), nan_code(kv_dtype) if poison else 0, dtype=store_dt)
    v_cache = np.full((NB, hkv, d, BS), nan_code(kv_dtype) if poison else 0, dtype=store_dt)
    kv_scales = np.ones((2, NB, hkv), dtype=np.float32)
    if poison:
        kv_scales[:, perm[used:]] = np.nan
    K64, V64 = [], []
    for b in range(B):
        L = int(lens[b])
        kraw = draw(key_fn, (L, hkv, d))
        vraw = draw(value_fn, (L, hkv, d))
        Kb = np.zeros((L, hkv, d))
        Vb = np.zeros((L, hkv, d))
        for j in range(nblk[b]):
            p = table[b, j]
            t0, t1 = j * BS, min(L, (j + 1) * BS)
            n = t1 - t0
            for g in range(hkv):
                kt, vt = kraw[t0:t1, g, :], vraw[t0:t1, g, :]
                ks = vs = 1.0
                if kv_dtype == "fp8_e4m3":
                    # a power-of-two-free scale so the dequantised values are not
                    # themselves fp8 codes
                    ks = float(np.float32(np.abs(kt).max() / 448.0 * fp8_headroom + 1e-30))
                    vs = float(np.float32(np.abs(vt).max() / 448.0 * fp8_headroom + 1e-30))
                    kv_scales[0, p, g] = ks
                    kv_scales[1, p, g] = vs
                kst, k64 = _store(kt / ks, kv_dtype)
                vst, v64 = _store(vt / vs, kv_dtype)
                k_cache[p, g, :n, :] = kst
                v_cache[p, g, :, :n] = vst.T
                Kb[t0:t1, g, :] = k64 * ks
                Vb[t0:t1, g, :] = v64 * vs
        K64.append(Kb)
        V64.append(Vb)
    return Case(q, q64, k_cache, v_cache, table, lens, kv_scales, K64, V64,
                q_dtype, kv_dtype, float(softmax_scale))
