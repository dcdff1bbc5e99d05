"""GPU parity of the shared-prefix decode path (GRPO groups whose samples'
block tables share the prompt's blocks) against the fp64 oracle of plain
paged attention: reading a shared block once for several members' queries
must not change the result. Tolerances as in test_parity_gpu."""

import time

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


def grpo(name, prompts, samples, Hq, Hkv, D, kv, plen=(150, 900), resp=(300, 1.0, 1500), cfg=60):
    return W.Workload(name, prompts * samples, Hq, Hkv, D, "bf16", kv,
                      ("grpo", prompts, samples, plen[0], plen[1], resp[0], resp[1], resp[2]), cfg_id=cfg)


def run_shared(lib, inp, group_size, shared_blocks, **opts):
    out = torch.empty_like(inp.q)
    sb = torch.as_tensor(np.asarray(shared_blocks, dtype=np.int32), device=DEV)
    lib.paged_decode_attention_shared_prefix(inp.q, inp.k_cache, inp.v_cache, inp.block_table, inp.seq_lens,
                                             inp.kv_scales, out, inp.softmax_scale, group_size, sb,
                                             max_seq_len=inp.layout.max_seq_len, **opts)
    torch.cuda.synchronize()
    return out


SPLITS = {
    "auto": {},
    "many_partials": {"waves_per_cu": 1, "min_blocks_per_wave": 1},
    "dynamic": {"chunks_per_wave": 16, "min_blocks_per_chunk": 1, "min_blocks_per_wave": 1, "waves_per_cu": 1},
}

# (prompts, samples, Hq, Hkv, D, kv): G = 1, 2, 4, 7, 8, 16 (M = 32, 16, 8, 4, 4, 2 members per
# prefix entry), groups smaller and larger than M (ragged last entry), group size 1.
CASES = [
    (2, 8, 32, 8, 128, "bf16"),
    (3, 5, 28, 4, 128, "bf16"),
    (2, 17, 8, 4, 64, "bf16"),
    (4, 3, 4, 4, 64, "bf16"),
    (2, 8, 64, 8, 128, "fp8_e4m3"),
    (3, 4, 32, 2, 64, "fp8_e4m3"),
    (5, 1, 8, 2, 128, "bf16"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}x{c[1]}_G{c[2] // c[3]}_D{c[4]}_{c[5]}")
def test_shared_prefix_matches_oracle(lib, case):
    prompts, samples, hq, hkv, d, kv = case
    w = grpo(f"sp_{prompts}x{samples}_{hq}_{hkv}_{d}_{kv}", prompts, samples, hq, hkv, d, kv)
    inp = W.generate(w, DEV)
    gs, sb = W.group_prefix(w, inp.layout)
    assert gs == samples and sb.max() > 0
    ref = U.oracle_for(inp)
    first = None
    for name, split in SPLITS.items():
        print(f"[parity] shared-prefix {w.name} split={name}", flush=True)
        got = run_shared(lib, inp, gs, sb, **split)
        U.assert_close(U.out_to_f64(got), ref, kv, f"{w.name} {name}")
        if name == "auto":
            first = got
            again = run_shared(lib, inp, gs, sb, **split)
            assert torch.equal(first.view(torch.int16), again.view(torch.int16)), "must be reproducible"
    assert lib.read_device_status() == 0


def test_shared_prefix_bounds_are_checked(lib):
    """A bound larger than what the members share (ids differ after the prompt,
    or a member is shorter), zero, or negative still gives the plain result; a
    bound that ids contradict is flagged (status bit 4)."""
    w = grpo("sp_bounds", 3, 6, 32, 8, 128, "bf16")
    inp = W.generate(w, DEV)
    gs, sb = W.group_prefix(w, inp.layout)
    ref = U.oracle_for(inp)
    full = (inp.layout.seq_lens // 16).reshape(-1, gs).min(axis=1)   # every member's full blocks
    for bound in (sb + 3, sb * 0 + 10 ** 6, sb * 0, sb * 0 - 5, sb):
        print(f"[parity] shared-prefix bounds {bound.tolist()}", flush=True)
        got = run_shared(lib, inp, gs, bound)
        U.assert_close(U.out_to_f64(got), ref, "bf16", f"bounds {bound.tolist()}")
        status = lib.read_device_status()
        # the members' ids agree exactly on the prompt's full blocks (sb), so a
        # bound is contradicted iff it still exceeds sb after the length clamp
        flagged = bool((np.minimum(np.maximum(bound, 0), full) > sb).any())
        assert bool(status & 4) == flagged, (bound.tolist(), status)
        assert status & 3 == 0


def test_shared_prefix_without_shared_blocks(lib):
    """Groups over a plain (unshared) layout: the ids differ from block 0 on,
    so every group falls back to private reads (the second group, whose
    members all have a full block, is flagged); empty sequences give zeros."""
    lens = [1, 17, 0, 300, 64, 33, 512, 20, 16, 100, 0, 45]
    w = W.Workload("sp_plain", len(lens), 16, 4, 128, "bf16", "bf16", ("uniform", 1, 1), cfg_id=61)
    inp = W.generate(w, DEV, seq_lens=lens)
    ref = U.oracle_for(inp)
    got = run_shared(lib, inp, 4, [5, 5, 5])
    U.assert_close(U.out_to_f64(got), ref, "bf16", "unshared layout")
    assert np.array_equal(U.out_to_f64(got)[2], np.zeros_like(ref[2]))
    assert lib.read_device_status() & 4


@pytest.mark.parametrize("name", ["grpo_bf16", "grpo_longprompt_bf16"])
def test_shared_prefix_full_size_grpo(lib, name):
    """The full GRPO steps through the shared-prefix path: every output (all
    B x Hq x D) against the oracle, whose sequences run in a pool of worker
    processes."""
    w = W.WORKLOADS[name]
    t0 = time.perf_counter()
    print(f"[parity] shared-prefix full {name}: generating", flush=True)
    inp = W.generate(w, DEV)
    gs, sb = W.group_prefix(w, inp.layout)
    got = U.out_to_f64(run_shared(lib, inp, gs, sb))
    assert lib.read_device_status() == 0
    ref = U.oracle_whole(inp, f"shared-prefix full {name}")
    max_abs, rel_l2 = U.assert_close(got, ref, "bf16", f"full {name} shared")
    worst, at = U.worst_row_rel_l2(got, ref)
    print(f"[parity] shared-prefix full {name}: all {got.size} outputs: max_abs {max_abs:.2e} rel_l2 {rel_l2:.2e}, "
          f"worst row rel_l2 {worst:.2e} at {tuple(int(i) for i in at)}; {time.perf_counter() - t0:.1f} s",
          flush=True)
    del inp
    torch.cuda.empty_cache()
