"""The decode entry point that allocates nothing
(pda_paged_decode_attention_noalloc), called through the C interface, against
the allocating pda_paged_decode_attention: the same kernels on the same
inputs, so the outputs must agree bit for bit, and both within the oracle's
bounds. The fixed scratch keeps the last call's contents, so calls are made in
a row with a smaller input second; a capture into a HIP graph comes first, so
that in a fresh process the capture is the entry point's first call."""

import numpy as np
import pytest
import torch

from paper_2605_20863_amd import workloads as W
from tests import _gpu_util as U

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a HIP device")
    from paper_2605_20863_amd import _lib
    return _lib


def bits(t):
    return t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32)


def call(lib, inp, noalloc, out=None, **opts):
    out = torch.empty_like(inp.q) if out is None else out
    fn = lib.paged_decode_attention_noalloc if noalloc else lib.paged_decode_attention
    fn(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens, inp.kv_scales, out, inp.softmax_scale,
       max_seq_len=inp.layout.max_seq_len, **opts)
    return out


def test_noalloc_graph_capture(lib):
    """Captured into a graph (the process's first no-allocation call when this
    file runs alone) and replayed with new queries written in place between
    replays: every replay equals the allocating call bit for bit."""
    inp = W.generate(W.SMALL_WORKLOADS["gqa7b_bf16"], DEV)
    out_g = torch.empty_like(inp.q)
    s = torch.cuda.Stream(DEV)
    g = torch.cuda.CUDAGraph()
    print("[noalloc] capturing", flush=True)
    with torch.cuda.graph(g, stream=s):
        call(lib, inp, True, out_g, waves_per_cu=16, min_blocks_per_wave=1)
    ref = U.oracle_for(inp)
    for r in range(3):
        with torch.cuda.stream(s):
            if r:
                gen = torch.Generator(device=DEV).manual_seed(100 + r)
                inp.q.copy_(torch.randn(inp.q.shape, generator=gen, device=DEV).to(inp.q.dtype))
            g.replay()
            out_e = call(lib, inp, False, waves_per_cu=16, min_blocks_per_wave=1)
        torch.cuda.synchronize()
        print(f"[noalloc] replay {r}", flush=True)
        assert torch.equal(bits(out_g), bits(out_e)), f"replay {r} differs from the allocating call"
        if r == 0:
            U.assert_close(U.out_to_f64(out_g), ref, "bf16", "noalloc graph replay")
    assert lib.read_device_status() == 0


CASES = [
    # (workload, lengths of the first call, lengths of the second, smaller call, options)
    ("fp8kv", None, [700, 3, 0, 129], {}),
    ("gqa7b_bf16", None, [40, 17], {"waves_per_cu": 16, "min_blocks_per_wave": 1}),
    ("straggler_bf16", None, [1500], {"chunks_per_wave": 4, "min_blocks_per_chunk": 1, "min_blocks_per_wave": 1}),
]


@pytest.mark.parametrize("name,first,second,opts", CASES, ids=[c[0] for c in CASES])
def test_noalloc_two_calls_second_smaller(lib, name, first, second, opts):
    w = W.SMALL_WORKLOADS[name]
    for i, lens in enumerate((first, second)):
        inp = W.generate(w, DEV, seq_lens=lens)
        print(f"[noalloc] {name} call {i}: {len(inp.layout.seq_lens)} sequences, opts {opts}", flush=True)
        got = call(lib, inp, True, **opts)
        ref_call = call(lib, inp, False, **opts)
        torch.cuda.synchronize()
        assert torch.equal(bits(got), bits(ref_call)), f"{name} call {i}: differs from the allocating call"
        U.assert_close(U.out_to_f64(got), U.oracle_for(inp), w.kv_dtype, f"noalloc {name} call {i}")
        if lens is not None and 0 in lens:
            assert not U.out_to_f64(got)[lens.index(0)].any(), "an empty sequence gives zeros"
    assert lib.read_device_status() == 0


def test_noalloc_full_size_fp8_step(lib):
    """The largest decode step (fp8 KV, 512 sequences, 64 / 8 heads) fits the
    fixed scratch at the default split: bit for bit the allocating call, then
    a smaller step (the 7B GQA step) right after it."""
    for name in ("fp8kv", "gqa7b_bf16"):
        inp = W.generate(W.WORKLOADS[name], DEV)
        print(f"[noalloc] full {name}", flush=True)
        got = call(lib, inp, True)
        ref_call = call(lib, inp, False)
        torch.cuda.synchronize()
        assert torch.equal(bits(got), bits(ref_call)), f"full {name}: differs from the allocating call"
        assert torch.isfinite(got.float()).all()
        del inp, got, ref_call
        torch.cuda.empty_cache()
    assert lib.read_device_status() == 0


def test_noalloc_rejects_calls_beyond_the_scratch(lib):
    """A split whose workspace exceeds the fixed array is refused with
    PDA_EINVAL before any launch; the next call that fits runs normally."""
    inp = W.generate(W.SMALL_WORKLOADS["fp8kv"], DEV)
    big = {"waves_per_cu": 64, "chunks_per_wave": 64}
    info = lib.query_plan(lib.problem_for(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens),
                          lib.make_options(**big))
    assert info.workspace_bytes > lib.NOALLOC_SCRATCH_BYTES
    with pytest.raises(lib.PdaError) as e:
        call(lib, inp, True, **big)
    assert e.value.code == lib.EINVAL and "fixed scratch" in str(e.value)
    got = call(lib, inp, True)
    torch.cuda.synchronize()
    U.assert_close(U.out_to_f64(got), U.oracle_for(inp), "fp8_e4m3", "noalloc after a refused call")
    assert lib.read_device_status() == 0
