"""The prefill attention kernel issues its direct global-to-LDS loads as inline
assembly that sets M0 (the LDS address of the load) itself. M0 is a register
the compiler reserves: these tests compile the prefill source for gfx950 with
the library's flags and check, in the generated assembly of every attention
kernel, that each write to M0 is immediately followed by the load that reads
it, and that no other instruction touches M0, so nothing the compiler emits
can depend on an M0 value the asm replaced. Host-only (hipcc cross-compiles).
"""

import os
import re
import subprocess

import pytest

from paper_2605_20863_amd import build as B

SRC = os.path.join(B.CSRC, "pda_prefill.hip")


@pytest.fixture(scope="module")
def prefill_asm(tmp_path_factory):
    try:
        hipcc = B.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("isa") / "pda_prefill.s"
    cmd = [hipcc, f"--offload-arch={B.ARCH}", "-O3", "-std=c++17", "-I", os.path.join(B.ROOT, "include"),
           "-I", B.CSRC, *B.HIP_FLAGS, *B.SOURCE_FLAGS.get("pda_prefill.hip", []), "--cuda-device-only", "-S",
           SRC, "-o", str(out)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    return out.read_text()


def kernels(asm):
    """{symbol: [instruction lines]} of every prefill attention kernel."""
    out, cur = {}, None
    for line in asm.splitlines():
        m = re.match(r"^(_Z\S*prefill_kernel\S*):", line)
        if m:
            cur = m.group(1)
            out[cur] = []
            continue
        if cur is None:
            continue
        s = line.split(";")[0].strip()
        if not s or s.startswith(".") or s.endswith(":"):
            continue
        out[cur].append(s)
        if s.startswith("s_endpgm"):
            cur = None
    return out


def test_every_m0_write_feeds_a_direct_load(prefill_asm):
    ks = kernels(prefill_asm)
    assert len(ks) == 8, sorted(ks)  # 2 cache dtypes x 2 head dims x (image, staging)
    image = 0
    for name, ins in ks.items():
        m0 = [i for i, s in enumerate(ins) if re.search(r"\bm0\b", s)]
        loads = [i for i, s in enumerate(ins) if s.startswith("global_load_lds")]
        for i in m0:
            assert ins[i].startswith("s_mov_b32 m0, "), (name, ins[i])
            assert ins[i + 1].startswith("global_load_lds"), (name, ins[i], ins[i + 1])
        assert len(m0) == len(loads), (name, len(m0), len(loads))
        if loads:
            image += 1
    assert image == 4  # only the image path loads directly


def test_no_other_reads_of_m0(prefill_asm):
    """Instructions that read M0 implicitly (indexed register moves, GWS,
    messages, interpolation) do not appear in the attention kernels."""
    implicit = re.compile(r"^(s_movrel|v_movrel|s_set_gpr_idx|ds_gws|s_sendmsg|v_interp|ds_append|ds_consume)")
    for name, ins in kernels(prefill_asm).items():
        bad = [s for s in ins if implicit.match(s)]
        assert not bad, (name, bad[:5])
