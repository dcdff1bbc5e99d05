"""Build the HIP library ``libpda.so`` in place for gfx950.

    python -m paper_2605_20863_amd.build

compiles every source under ``csrc/`` with hipcc (one object per source, in
parallel) and links ``paper_2605_20863_amd/libpda.so`` (written to a temporary
name, then renamed, so a concurrent loader never sees a half-written file).
"""

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libpda.so")

SOURCES = ["pda_kernels.hip", "pda_append.hip", "pda_prefill.hip", "pda_scratch.hip", "pda_host.cpp"]
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


# Per-source device flags. The prefill kernels never rely on NaN semantics
# (dead cache slots are masked bitwise, masked logits are -inf), so they run
# with IEEE mode off: max and min then need no NaN-quieting copies. (The decode
# source gains nothing from it and its G = 8 vector kernels then spill.)
SOURCE_FLAGS = {
    "pda_prefill.hip": ["-Xarch_device", "-fno-honor-nans", "-Xarch_device", "-mno-amdgpu-ieee"],
}


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 target feature; that note is harmless
    noise = "is not a recognized feature for this target"
    log = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{log}")
    if verbose and log.strip():
        print(log)


def build(verbose: bool = False) -> str:
    """Compile every source to an object (in parallel), then link libpda.so."""
    import tempfile
    from concurrent.futures import ThreadPoolExecutor

    out_tmp = LIB + f".tmp{os.getpid()}"
    link = []
    rt = hip_runtime_dir()
    if rt:
        link = ["-L", rt, f"-Wl,-rpath,{rt}"]
    common = [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
              "-I", os.path.join(ROOT, "include"), "-I", CSRC, *HIP_FLAGS]
    with tempfile.TemporaryDirectory(prefix="pda_build_") as tmp:
        objs = [os.path.join(tmp, s + ".o") for s in SOURCES]
        cmds = [[*common, *SOURCE_FLAGS.get(s, []), "-c", os.path.join(CSRC, s), "-o", o]
                for s, o in zip(SOURCES, objs)]
        with ThreadPoolExecutor(max_workers=len(cmds)) as pool:
            for f in [pool.submit(_run, c, verbose) for c in cmds]:
                f.result()
        try:
            _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, *link, "-o", out_tmp], verbose)
        except Exception:
            if os.path.exists(out_tmp):
                os.unlink(out_tmp)
            raise
    os.replace(out_tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
