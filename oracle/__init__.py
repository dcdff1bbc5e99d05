"""CPU fp64 oracle for paged-KV decode attention.

TEST INFRASTRUCTURE ONLY. Nothing in the product path (the package
``paper_2605_20863_amd``, its HIP library or its Python binding) may import,
call, link or execute anything under ``oracle/``. Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` use it.

The oracle is deliberately plain and slow: numpy in float64, one sequence and
one KV head at a time, no blocking, no fusion, no reordering beyond the
definition it restates. It shares no code with the GPU path: it has its own
bfloat16 and OCP FP8 E4M3 decoders and reads the paged cache through its own
indexing.

What it computes. The paper (Sec. 2.2) identifies rollout decoding -- one new
token per live sequence per step, over a long-tailed length mix -- as the
phase whose throughput collapses in the tail, and Sec. 6.2 / Fig. e2e-conv(c)
reports decode throughput per GPU. Each decode step of a Transformer (the
architecture family named in Sec. 1, Vaswani et al. 2017, Eq. 1 there) attends
the new token's query to the keys and values cached for its sequence:

    out[b, h, :] = softmax(scale * K_b q[b, h]) V_b

with K_b, V_b the sequence's cached keys/values for KV head h // G, read
through a block table as in the paged KV-cache memory management the paper
cites in Sec. 8 (vLLM / PagedAttention).

``kv_append`` restates the step before it: writing each sequence's new key and
value into its paged cache, with the fp8 tile-scale policy the library uses.
"""

from .decode_attention import (  # noqa: F401
    DTYPES,
    bf16_to_f64,
    e4m3fn_to_f64,
    decode,
    gather_sequence,
    paged_decode_attention,
    paged_multi_token_attention,
    paged_prefill_attention,
    attend,
    attend_partial,
    combine_partials,
)
from .kv_append import encode_bf16, encode_e4m3fn, append_tile_fp8, paged_kv_append  # noqa: F401,E402
