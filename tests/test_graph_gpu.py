"""The library's calls inside HIP graphs: once a stream's workspace is large
enough a call enqueues kernel launches only, so a decode step (or a whole
append + decode step of a serving loop) can be captured once and replayed.

Every test replays a captured call several times with eager work and
synchronisation between the replays (inputs changed in place), and checks
every replay bit for bit against the same call made eagerly, plus the first
against the fp64 oracle. The calls are deterministic (the split does not
change the result), so equality is exact."""

import numpy as np
import pytest
import torch

import oracle

from paper_2605_20863_amd import workloads as W
from tests import _gpu_util as U

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
REPLAYS = 3


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    from paper_2605_20863_amd import _lib
    return _lib


def bits(t):
    return t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32)


def fresh_q(q, seed):
    g = torch.Generator(device=DEV).manual_seed(seed)
    return torch.randn(q.shape, generator=g, device=DEV).to(q.dtype)


def replay_and_compare(call, out_g, out_e, mutate, check_first):
    """Warm the stream's workspace eagerly, capture call(out_g), then for each
    replay: mutate the inputs in place, replay, run call(out_e) eagerly, and
    compare bit for bit."""
    s = torch.cuda.Stream(DEV)
    with torch.cuda.stream(s):
        call(out_e)
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        call(out_g)
    for r in range(REPLAYS):
        with torch.cuda.stream(s):
            mutate(r)
            g.replay()
            call(out_e)
        torch.cuda.synchronize()
        print(f"[graph] replay {r}", flush=True)
        assert torch.equal(bits(out_g), bits(out_e)), f"replay {r} differs from the eager call"
        if r == 0:
            check_first(out_g)


DECODE_CASES = {
    "gqa7b_bf16": (W.SMALL_WORKLOADS["gqa7b_bf16"], {}),
    "gqa7b_bf16_dynamic": (W.SMALL_WORKLOADS["gqa7b_bf16"],
                           {"chunks_per_wave": 8, "min_blocks_per_chunk": 1, "min_blocks_per_wave": 1}),
    "tiny_mha_f32_vector": (W.SMALL_WORKLOADS["tiny_mha_f32"], {}),
    "fp8kv": (W.SMALL_WORKLOADS["fp8kv"], {}),
}


@pytest.mark.parametrize("name", list(DECODE_CASES))
def test_graph_decode(lib, name):
    w, opts = DECODE_CASES[name]
    inp = W.generate(w, DEV)
    out_g, out_e = torch.empty_like(inp.q), torch.empty_like(inp.q)

    def call(out):
        lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, inp.kv_scales,
                                   out, inp.softmax_scale, max_seq_len=inp.layout.max_seq_len, **opts)

    def mutate(r):
        inp.q.copy_(fresh_q(inp.q, 100 + r))

    replay_and_compare(call, out_g, out_e, mutate,
                       lambda out: U.assert_close(U.out_to_f64(out), U.oracle_for(inp), w.kv_dtype, f"graph {name}"))
    assert lib.read_device_status() == 0


def test_graph_multi_token_two_tiles(lib):
    """4 query tokens on the 7B shape (28 columns, the two-tile body and two
    combine workgroups per unit)."""
    w = W.SMALL_WORKLOADS["gqa7b_bf16"].replace(name="graph_spec4", q_tokens=4)
    inp = W.generate(w, DEV)
    assert inp.q.dim() == 4
    out_g, out_e = torch.empty_like(inp.q), torch.empty_like(inp.q)

    def call(out):
        lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, inp.kv_scales,
                                   out, inp.softmax_scale, max_seq_len=inp.layout.max_seq_len)

    def check(out):
        lay = inp.layout
        ref = oracle.paged_multi_token_attention(
            q=U.raw(inp.q), k_cache=U.raw(inp.k_cache), v_cache=U.raw(inp.v_cache), block_table=lay.block_table,
            seq_lens=lay.seq_lens, softmax_scale=inp.softmax_scale, q_dtype="bf16", kv_dtype="bf16")
        U.assert_close(U.out_to_f64(out), ref, "bf16", "graph multi-token", bf16_out_rounding=True)

    replay_and_compare(call, out_g, out_e, lambda r: inp.q.copy_(fresh_q(inp.q, 200 + r)), check)
    assert lib.read_device_status() == 0


def test_graph_shared_prefix(lib):
    w = W.SMALL_WORKLOADS["grpo_bf16"]
    inp = W.generate(w, DEV)
    gs, sb = W.group_prefix(w, inp.layout)
    sbd = torch.as_tensor(np.asarray(sb, dtype=np.int32), device=DEV)
    out_g, out_e = torch.empty_like(inp.q), torch.empty_like(inp.q)

    def call(out):
        lib.paged_decode_attention_shared_prefix(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                                                 inp.kv_scales, out, inp.softmax_scale, gs, sbd,
                                                 max_seq_len=inp.layout.max_seq_len)

    replay_and_compare(call, out_g, out_e, lambda r: inp.q.copy_(fresh_q(inp.q, 300 + r)),
                       lambda out: U.assert_close(U.out_to_f64(out), U.oracle_for(inp), "bf16", "graph shared"))
    assert lib.read_device_status() == 0


def test_graph_prefill(lib):
    w = W.WORKLOADS["logprob_gqa7b_bf16"].replace(name="graph_logprob", num_seqs=5,
                                                  lengths=("lognormal", 150, 0.8, 1, 400))
    pin = W.generate_prefill(w, DEV)
    c = pin.cache
    out_g = torch.empty(pin.q.shape, dtype=torch.bfloat16, device=DEV)
    out_e = torch.empty_like(out_g)

    def call(out):
        lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, c.v_cache, c.block_table, c.seq_lens, None,
                                    out, c.softmax_scale, max_seq_len=c.layout.max_seq_len)

    def check(out):
        ref = oracle.paged_prefill_attention(
            q=U.raw(pin.q), q_offsets=pin.offsets, k_cache=U.raw(c.k_cache), v_cache=U.raw(c.v_cache),
            block_table=c.layout.block_table, seq_lens=c.layout.seq_lens, softmax_scale=c.softmax_scale,
            q_dtype="bf16", kv_dtype="bf16")
        U.assert_close(U.out_to_f64(out), ref, "bf16", "graph prefill", bf16_out_rounding=True)

    replay_and_compare(call, out_g, out_e, lambda r: pin.q.copy_(fresh_q(pin.q, 400 + r)), check)
    assert lib.read_device_status() == 0


def test_graph_prefill_more_units_than_workgroups(lib):
    """Enough tiles that the persistent grid claims most units from its queue
    counters: the plan kernel must reset them on every replay (a stale counter
    would skip units, which the oracle check of the first replay, made after an
    eager call on the same stream, would show)."""
    w = W.WORKLOADS["logprob_gqa7b_bf16"].replace(name="graph_logprob_many", num_seqs=24,
                                                  lengths=("lognormal", 600, 0.5, 64, 1500))
    pin = W.generate_prefill(w, DEV)
    c = pin.cache
    units = sum((int(n) + 35) // 36 for n in pin.counts) * w.num_kv_heads
    assert units > 4 * torch.cuda.get_device_properties(DEV).multi_processor_count, units
    out_g = torch.empty(pin.q.shape, dtype=torch.bfloat16, device=DEV)
    out_e = torch.empty_like(out_g)

    def call(out):
        lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, c.v_cache, c.block_table, c.seq_lens, None,
                                    out, c.softmax_scale, max_seq_len=c.layout.max_seq_len)

    def check(out):
        ref = U.oracle_prefill_whole(pin, "graph prefill, many units")
        U.assert_close(U.out_to_f64(out), ref, "bf16", "graph prefill, many units", bf16_out_rounding=True)

    replay_and_compare(call, out_g, out_e, lambda r: pin.q.copy_(fresh_q(pin.q, 500 + r)), check)
    assert lib.read_device_status() == 0


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_graph_prefill_capture_falls_back_to_staging(lib, monkeypatch, kv):
    """A stream whose workspace was sized by a staging-path call (image cap 0)
    is captured with the image allowed again: a capture cannot grow the
    workspace for the image, so the recorded call converts tiles in registers.
    Every replay matches an eager image-path call on another stream bit for
    bit, and the first matches the oracle."""
    w = W.WORKLOADS["logprob_gqa7b_bf16"].replace(name=f"graph_prefill_staging_{kv}", num_seqs=6, kv_dtype=kv,
                                                  lengths=("lognormal", 300, 0.5, 16, 700))
    pin = W.generate_prefill(w, DEV)
    c = pin.cache
    out_g = torch.empty(pin.q.shape, dtype=torch.float32, device=DEV)
    out_e = torch.empty_like(out_g)

    def call(out):
        lib.paged_prefill_attention(pin.q, pin.q_offsets, c.k_cache, c.v_cache, c.block_table, c.seq_lens,
                                    c.kv_scales, out, c.softmax_scale, max_seq_len=c.layout.max_seq_len)

    s = torch.cuda.Stream(DEV)
    monkeypatch.setenv("PDA_PREFILL_IMAGE_MAX_MB", "0")
    with torch.cuda.stream(s):
        call(out_g)  # sizes this stream's workspace for the staging path only
    s.synchronize()
    monkeypatch.delenv("PDA_PREFILL_IMAGE_MAX_MB")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        call(out_g)
    for r in range(REPLAYS):
        with torch.cuda.stream(s):
            pin.q.copy_(fresh_q(pin.q, 700 + r))
            g.replay()
        s.synchronize()
        call(out_e)  # the current stream: its own workspace, room for the image
        torch.cuda.synchronize()
        print(f"[graph] replay {r}", flush=True)
        assert torch.equal(bits(out_g), bits(out_e)), f"replay {r} differs from the eager image-path call"
        if r == 0:
            ref = U.oracle_prefill_whole(pin, f"graph prefill staging {kv}")
            U.assert_close(U.out_to_f64(out_g), ref, kv, f"graph prefill staging {kv}")
    assert lib.read_device_status() == 0


@pytest.mark.parametrize("kv", ["bf16", "fp8_e4m3"])
def test_graph_append_decode_loop(lib, kv):
    """A serving loop as one graph: append each sequence's new key and value
    at its position, then attend with the new length. Positions and lengths
    advance in place between replays; a twin cache runs the same steps eagerly
    and must match bit for bit after every step (cache, fp8 scales, output)."""
    rng = np.random.default_rng(77)
    B, hkv, G, d, maxb = 6, 2, 4, 128, 6
    NB = B * maxb + 4
    table = torch.from_numpy(rng.permutation(NB)[:B * maxb].reshape(B, maxb).astype(np.int32)).to(DEV)
    lens0 = rng.integers(1, 16 * maxb - 8, B).astype(np.int32)
    dt = torch.bfloat16 if kv == "bf16" else torch.uint8
    if kv == "bf16":
        k0 = torch.randn((NB, hkv, 16, d), device=DEV).to(dt)
        v0 = torch.randn((NB, hkv, d, 16), device=DEV).to(dt)
        s0 = None
    else:  # codes of magnitude <= 1 (no NaN patterns), unit scales
        k0 = torch.randint(0, 0x38, (NB, hkv, 16, d), device=DEV, dtype=torch.uint8)
        v0 = torch.randint(0, 0x38, (NB, hkv, d, 16), device=DEV, dtype=torch.uint8)
        s0 = torch.ones((2, NB, hkv), device=DEV)
    caches = {t: (k0.clone(), v0.clone(), s0.clone() if s0 is not None else None) for t in ("graph", "eager")}
    outs = {t: torch.empty((B, hkv * G, d), dtype=torch.bfloat16, device=DEV) for t in ("graph", "eager")}
    # the new token goes to slot L of a sequence holding L tokens, which then holds L + 1
    positions = torch.from_numpy(lens0.copy()).to(DEV)
    seq_lens = torch.from_numpy(lens0 + 1).to(DEV)
    k_new = torch.empty((B, hkv, d), dtype=torch.bfloat16, device=DEV)
    v_new = torch.empty_like(k_new)
    q = torch.empty((B, hkv * G, d), dtype=torch.bfloat16, device=DEV)

    def fill(step):
        g = torch.Generator(device=DEV).manual_seed(500 + step)
        for t in (k_new, v_new, q):
            t.copy_(torch.randn(t.shape, generator=g, device=DEV).to(t.dtype))

    def step_call(which):
        kc, vc, sc = caches[which]
        lib.paged_kv_append(k_new, v_new, kc, vc, sc, table, positions)
        lib.paged_decode_attention(q, kc, vc, table, seq_lens, sc, outs[which], d ** -0.5, max_seq_len=16 * maxb)

    s = torch.cuda.Stream(DEV)
    fill(0)
    with torch.cuda.stream(s):
        step_call("eager")
        step_call("graph")  # the same step on the graph's cache, so both twins hold the same state
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        step_call("graph")
    for step in range(1, 6):
        with torch.cuda.stream(s):
            positions.add_(1)
            seq_lens.add_(1)
            fill(step)
            g.replay()
            step_call("eager")
        torch.cuda.synchronize()
        print(f"[graph] serving step {step}", flush=True)
        for a, b in zip(caches["graph"], caches["eager"]):
            if a is not None:
                assert torch.equal(a.view(torch.uint8), b.view(torch.uint8)), f"step {step}: caches differ"
        assert torch.equal(bits(outs["graph"]), bits(outs["eager"])), f"step {step}: outputs differ"
    kc, vc, sc = caches["graph"]
    ref = oracle.paged_decode_attention(q=U.raw(q), k_cache=U.raw(kc), v_cache=U.raw(vc),
                                        block_table=U.raw(table), seq_lens=U.raw(seq_lens), softmax_scale=d ** -0.5,
                                        q_dtype="bf16", kv_dtype=kv, kv_scales=U.raw(sc) if sc is not None else None)
    U.assert_close(U.out_to_f64(outs["graph"]), ref, kv, f"graph serving loop {kv}")
    assert lib.read_device_status() == 0


def test_graph_survives_workspace_growth(lib):
    """A graph captured on a stream stays valid after a larger eager call on
    that stream grows its workspace (the old allocation is kept for it)."""
    small = W.generate(W.SMALL_WORKLOADS["gqa7b_bf16"], DEV)
    big = W.generate(W.SMALL_WORKLOADS["fp8kv"], DEV)
    s = torch.cuda.Stream(DEV)
    out_g, out_e, out_big = torch.empty_like(small.q), torch.empty_like(small.q), torch.empty_like(big.q)
    many = {"waves_per_cu": 16, "chunks_per_wave": 8, "min_blocks_per_chunk": 1, "min_blocks_per_wave": 1}

    def call(inp, out, **opts):
        lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, inp.kv_scales,
                                   out, inp.softmax_scale, max_seq_len=inp.layout.max_seq_len, **opts)

    with torch.cuda.stream(s):
        call(small, out_e)
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        call(small, out_g)
    with torch.cuda.stream(s):
        call(big, out_big, **many)  # needs far more partial slots: the workspace grows
    s.synchronize()
    U.assert_close(U.out_to_f64(out_big), U.oracle_for(big), "fp8_e4m3", "after growth")
    for r in range(REPLAYS):
        with torch.cuda.stream(s):
            small.q.copy_(fresh_q(small.q, 600 + r))
            g.replay()
            call(small, out_e)
        torch.cuda.synchronize()
        assert torch.equal(bits(out_g), bits(out_e)), f"replay {r} after growth"
    assert lib.read_device_status() == 0


def test_capture_that_needs_growth_is_refused(lib):
    """Growing the workspace cannot be recorded: the call returns PDA_EINVAL
    (nothing is allocated or enqueued) and the stream stays usable."""
    # 4 query tokens of 7 heads with the most chunks the options allow: partial
    # rows of 28 columns for ~1M chunks, larger than any workspace grown before
    inp = W.generate(W.SMALL_WORKLOADS["gqa7b_bf16"].replace(name="graph_refused", q_tokens=4), DEV)
    out = torch.empty_like(inp.q)
    huge = {"waves_per_cu": 64, "chunks_per_wave": 64, "min_blocks_per_chunk": 1, "min_blocks_per_wave": 1}
    s = torch.cuda.Stream(DEV)
    g = torch.cuda.CUDAGraph()
    with pytest.raises(lib.PdaError, match="graph"):
        with torch.cuda.graph(g, stream=s):
            lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, None, out,
                                       inp.softmax_scale, max_seq_len=inp.layout.max_seq_len, **huge)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        lib.paged_decode_attention(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, None, out,
                                   inp.softmax_scale, max_seq_len=inp.layout.max_seq_len)
    torch.cuda.synchronize()
    lay = inp.layout
    ref = oracle.paged_multi_token_attention(
        q=U.raw(inp.q), k_cache=U.raw(inp.k_cache), v_cache=U.raw(inp.v_cache), block_table=lay.block_table,
        seq_lens=lay.seq_lens, softmax_scale=inp.softmax_scale, q_dtype="bf16", kv_dtype="bf16")
    U.assert_close(U.out_to_f64(out), ref, "bf16", "after a refused capture", bf16_out_rounding=True)
