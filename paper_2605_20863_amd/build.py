"""Build the HIP library ``libpda.so`` in place for gfx950.

    python -m paper_2605_20863_amd.build

compiles every source under ``csrc/`` with hipcc into
``paper_2605_20863_amd/libpda.so`` (written to a temporary name, then renamed,
so a concurrent loader never sees a half-written file).
"""

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libpda.so")

SOURCES = ["pda_kernels.hip", "pda_append.hip", "pda_prefill.hip", "pda_host.cpp"]
ARCH = "gfx950"

# No packed-FP32 instructions: they are kept out of every HIP object.
HIP_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc():
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def hip_runtime_dir():
    """Directory of the HIP runtime the process will already have loaded.

    PyTorch-ROCm ships its own libamdhip64.so (no SONAME). Linking against that
    copy records NEEDED "libamdhip64.so", which the dynamic loader resolves to
    the runtime torch has already mapped, so torch and this library share one
    HIP runtime (two runtimes in one process do not see the same device). Without
    torch, the library falls back to the ROCm installation's runtime.
    """
    import importlib.util

    spec = importlib.util.find_spec("torch")
    if spec and spec.submodule_search_locations:
        d = os.path.join(list(spec.submodule_search_locations)[0], "lib")
        if os.path.exists(os.path.join(d, "libamdhip64.so")):
            return d
    return None


def build(verbose: bool = False) -> str:
    out_tmp = LIB + f".tmp{os.getpid()}"
    link = []
    rt = hip_runtime_dir()
    if rt:
        link = ["-L", rt, f"-Wl,-rpath,{rt}"]
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-shared", "-fPIC",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, *HIP_FLAGS,
           *[os.path.join(CSRC, s) for s in SOURCES], *link, "-o", out_tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 target feature; that note is harmless
    noise = "is not a recognized feature for this target"
    log = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    if res.returncode != 0:
        if os.path.exists(out_tmp):
            os.unlink(out_tmp)
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{log}")
    if verbose and log.strip():
        print(log)
    os.replace(out_tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
