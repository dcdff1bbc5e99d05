"""MI355X (gfx950) paged-KV decode attention.

The product is the HIP library ``libpda.so`` behind the C interface in
``include/pda.h``; ``paper_2605_20863_amd._lib`` is its thin Python binding
and ``paper_2605_20863_amd.workloads`` draws seeded synthetic decode steps.
"""


def __getattr__(name):
    # Load the HIP library only when the binding is used, so the generators
    # and the build script stay importable before the library is built.
    if name in ("paged_decode_attention", "query_plan", "read_device_status",
                "release_workspaces", "version", "last_error", "PdaError"):
        from . import _lib
        return getattr(_lib, name)
    raise AttributeError(name)
