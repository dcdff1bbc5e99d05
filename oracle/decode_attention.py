"""fp64 reference for one batched paged-KV decode-attention step.

TEST INFRASTRUCTURE ONLY (see the package docstring): never imported by the
product path.

Data layout (the paper prescribes none; this is the layout the library's C
interface documents, restated here from the interface, not shared with it):

    q            [B, Hq, D]            f32 or bf16
    k_cache      [NB, Hkv, BS, D]      f32, bf16 or fp8 e4m3fn  (token-major tile)
    v_cache      [NB, Hkv, D, BS]      same dtype as k_cache    (dim-major tile)
    block_table  [B, max_blocks]       int32 physical block ids
    seq_lens     [B]                   int32
    kv_scales    [2, NB, Hkv]          fp32 dequant scales (index 0 = K, 1 = V),
                                       only for fp8 caches

Query head h reads KV head h // G with G = Hq // Hkv (contiguous grouping).
Token t of sequence b lives in physical block block_table[b, t // BS] at slot
t % BS. Slots t >= seq_lens[b] and block-table entries past the last used
block are never read.

Arrays for bf16 data hold the raw 16-bit patterns (uint16); fp8 arrays hold
the raw 8-bit codes (uint8); f32 arrays are float32.
"""

import math

import numpy as np

DTYPES = ("f32", "bf16", "fp8_e4m3")


def bf16_to_f64(bits):
    """Exact bfloat16 -> float64.

    bfloat16 is the upper half of an IEEE-754 binary32 pattern, so widening the
    16 stored bits to 32 (low half zero) gives the same number as a float32,
    which float64 represents exactly.
    """
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _e4m3fn_value(code):
    """Value of one OCP FP8 E4M3 ("fn": finite, no infinities) code.

    Layout S.EEEE.MMM, exponent bias 7. Exponent field 0 encodes subnormals
    (-1)^S * 2^(1-7) * M/8; the pattern S.1111.111 is NaN; every other code is
    (-1)^S * 2^(E-7) * (1 + M/8), so the largest finite magnitude is
    2^8 * 1.75 = 448 (OCP 8-bit floating point specification, E4M3).
    """
    s = (code >> 7) & 1
    e = (code >> 3) & 0xF
    m = code & 0x7
    sign = -1.0 if s else 1.0
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return sign * math.ldexp(m / 8.0, 1 - 7)
    return sign * math.ldexp(1.0 + m / 8.0, e - 7)


_E4M3FN_TABLE = np.array([_e4m3fn_value(c) for c in range(256)], dtype=np.float64)


def e4m3fn_to_f64(codes):
    """Exact OCP E4M3 (fn) -> float64 through the 256-entry table above."""
    codes = np.asarray(codes, dtype=np.uint8)
    return _E4M3FN_TABLE[codes]


def decode(arr, dtype):
    """Decode stored elements of ``dtype`` exactly to float64."""
    if dtype == "f32":
        return np.asarray(arr, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return bf16_to_f64(arr)
    if dtype == "fp8_e4m3":
        return e4m3fn_to_f64(arr)
    raise ValueError(f"unknown dtype {dtype!r}")


def gather_sequence(k_cache, v_cache, block_table, seq_len, b, g, kv_dtype, kv_scales=None):
    """Keys and values of sequence b, KV head g, as float64 [L, D] each.

    Walks the sequence's logical tokens t = 0..L-1, looks up the physical block
    block_table[b, t // BS] and the slot t % BS, decodes the stored elements and,
    for fp8 caches, multiplies by that block's per-(block, KV head) scale.
    """
    L = int(seq_len)
    nb, hkv, bs, d = k_cache.shape
    K = np.zeros((L, d), dtype=np.float64)
    V = np.zeros((L, d), dtype=np.float64)
    for t in range(0, L, bs):
        p = int(block_table[b, t // bs])
        if not (0 <= p < nb):
            raise IndexError(f"block_table[{b}, {t // bs}] = {p} outside [0, {nb})")
        n = min(bs, L - t)
        k_tile = decode(k_cache[p, g, :n, :], kv_dtype)          # [n, D]
        v_tile = decode(v_cache[p, g, :, :n], kv_dtype).T        # [D, n] -> [n, D]
        if kv_dtype == "fp8_e4m3":
            k_tile = k_tile * float(kv_scales[0, p, g])
            v_tile = v_tile * float(kv_scales[1, p, g])
        K[t:t + n] = k_tile
        V[t:t + n] = v_tile
    return K, V


def attend(qvec, K, V, softmax_scale):
    """softmax(scale * K q) V for one query vector; zeros when there are no keys.

    s_t = scale * <q, K_t>; subtracting m = max_t s_t leaves the softmax
    unchanged and keeps exp() in range; out = sum_t w_t V_t / sum_t w_t with
    w_t = exp(s_t - m).
    """
    if K.shape[0] == 0:
        return np.zeros(V.shape[1], dtype=np.float64)
    s = softmax_scale * (K @ qvec)
    m = np.max(s)
    w = np.exp(s - m)
    return (w @ V) / np.sum(w)


def attend_partial(qvec, K, V, softmax_scale):
    """Unnormalised softmax state (m, l, acc) of one query over a token subset.

    m = max_t s_t, l = sum_t exp(s_t - m), acc = sum_t exp(s_t - m) V_t, with
    s_t as in ``attend``. An empty subset gives (-inf, 0, 0).
    """
    d = V.shape[1]
    if K.shape[0] == 0:
        return -math.inf, 0.0, np.zeros(d, dtype=np.float64)
    s = softmax_scale * (K @ qvec)
    m = float(np.max(s))
    w = np.exp(s - m)
    return m, float(np.sum(w)), w @ V


def combine_partials(parts):
    """Merge (m, l, acc) states of disjoint token subsets into the attention output.

    With M = max_i m_i and c_i = exp(m_i - M), the union's sum of weights is
    sum_i c_i l_i and its weighted value sum is sum_i c_i acc_i (log-sum-exp
    rescaling); empty subsets (m = -inf) contribute nothing.
    """
    live = [(m, l, a) for (m, l, a) in parts if m != -math.inf]
    if not live:
        return np.zeros_like(parts[0][2])
    M = max(m for m, _, _ in live)
    num = sum(math.exp(m - M) * a for m, _, a in live)
    den = sum(math.exp(m - M) * l for m, l, _ in live)
    return num / den


def paged_decode_attention(q, k_cache, v_cache, block_table, seq_lens, softmax_scale,
                           q_dtype, kv_dtype, kv_scales=None, seqs=None):
    """Reference output of one decode step, float64 [len(seqs), Hq, D].

    For every sequence b (all of them, or the listed ``seqs``) and query head h:
    gather K, V of KV head h // G through the block table, then
    out[b, h] = softmax(scale * K q[b, h]) V.
    """
    B, hq, d = q.shape
    hkv = k_cache.shape[1]
    if hq % hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = hq // hkv
    if kv_dtype == "fp8_e4m3" and kv_scales is None:
        raise ValueError("fp8 caches need kv_scales")
    seqs = range(B) if seqs is None else list(seqs)
    qd = decode(q, q_dtype)
    out = np.zeros((len(seqs), hq, d), dtype=np.float64)
    for i, b in enumerate(seqs):
        for g in range(hkv):
            K, V = gather_sequence(k_cache, v_cache, block_table, seq_lens[b], b, g,
                                   kv_dtype, kv_scales)
            for h in range(g * G, (g + 1) * G):
                out[i, h] = attend(qd[b, h], K, V, softmax_scale)
    return out


def paged_multi_token_attention(q, k_cache, v_cache, block_table, seq_lens, softmax_scale,
                                q_dtype, kv_dtype, kv_scales=None, seqs=None):
    """Reference output of one step with Q new query tokens per sequence,
    float64 [len(seqs), Q, Hq, D].

    Speculative rollouts (named among RLVR rollout strategies in the paper's
    Sec. 1) verify several drafted tokens in one step: the cache already holds
    the Q new tokens as the last Q of the sequence's L, and query token i
    (0-based among the Q) sits at position L - Q + i, so causally it attends to
    tokens 0 .. L - Q + i. A query with no visible token (L - Q + i < 0) gives
    zeros. Q = 1 is the decode step above.
    """
    B, Q, hq, d = q.shape
    hkv = k_cache.shape[1]
    if hq % hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = hq // hkv
    if kv_dtype == "fp8_e4m3" and kv_scales is None:
        raise ValueError("fp8 caches need kv_scales")
    seqs = range(B) if seqs is None else list(seqs)
    qd = decode(q, q_dtype)
    out = np.zeros((len(seqs), Q, hq, d), dtype=np.float64)
    for n, b in enumerate(seqs):
        L = int(seq_lens[b])
        for g in range(hkv):
            K, V = gather_sequence(k_cache, v_cache, block_table, L, b, g, kv_dtype, kv_scales)
            for i in range(Q):
                visible = max(L - Q + i + 1, 0)
                for h in range(g * G, (g + 1) * G):
                    out[n, i, h] = attend(qd[b, i, h], K[:visible], V[:visible], softmax_scale)
    return out


def paged_prefill_attention(q, q_offsets, k_cache, v_cache, block_table, seq_lens, softmax_scale,
                            q_dtype, kv_dtype, kv_scales=None, seqs=None):
    """Reference output of a variable-length prefill over the paged cache,
    float64 [T, Hq, D] (rows of the listed ``seqs`` only when given; others 0).

    The log-prob forward of RLVR training (the compute_log_prob phase timed in
    the paper's Table 2, Sec. 6.3, one of the forward calls of its Sec. 4.2
    interface) and chunked prefill run attention for many query tokens per
    sequence at once. Packed q rows q_offsets[b] .. q_offsets[b + 1] - 1 are
    the last n_b tokens of sequence b (whose cache holds all L_b tokens), so
    query token i sits at position L_b - n_b + i and attends causally to
    tokens 0 .. L_b - n_b + i; a query with no visible token gives zeros.
    """
    T, hq, d = q.shape
    hkv = k_cache.shape[1]
    if hq % hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = hq // hkv
    if kv_dtype == "fp8_e4m3" and kv_scales is None:
        raise ValueError("fp8 caches need kv_scales")
    B = len(seq_lens)
    seqs = range(B) if seqs is None else list(seqs)
    qd = decode(q, q_dtype)
    out = np.zeros((T, hq, d), dtype=np.float64)
    for b in seqs:
        L = int(seq_lens[b])
        r0, r1 = int(q_offsets[b]), int(q_offsets[b + 1])
        n = r1 - r0
        for g in range(hkv):
            K, V = gather_sequence(k_cache, v_cache, block_table, L, b, g, kv_dtype, kv_scales)
            for i in range(n):
                visible = min(max(L - n + i + 1, 0), L)
                for h in range(g * G, (g + 1) * G):
                    out[r0 + i, h] = attend(qd[r0 + i, h], K[:visible], V[:visible], softmax_scale)
    return out
