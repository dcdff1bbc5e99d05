"""ctypes binding of the C interface in include/pda.h.

Argument marshalling only: every step of the decode attention, KV append and
prefill runs in the HIP library ``libpda.so``. Importing this module fails loudly when the
library has not been built; there is no fallback.

torch is used for device memory and streams: tensors provide device pointers
(``data_ptr()``) and the current HIP stream (``torch.cuda.current_stream()``).
"""

from __future__ import annotations

import ctypes
import os
import re

_PKG = os.path.dirname(os.path.abspath(__file__))
# PDA_LIBRARY may point at another build of the same library (same C interface)
LIB_PATH = os.environ.get("PDA_LIBRARY") or os.path.join(_PKG, "libpda.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "pda.h")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build the HIP library first "
        "(python -m paper_2605_20863_amd.build); there is no CPU fallback")

# Map PyTorch's bundled HIP runtime before the library: libpda.so then binds to
# that already-loaded runtime (same SONAME), so torch and the library share one
# HIP runtime instead of each bringing up its own (a second runtime in the
# process does not see the device).
try:
    import torch as _torch_rt  # noqa: F401
except ImportError:  # pure C-ABI use without torch: the ROCm installation's runtime
    _torch_rt = None

_lib = ctypes.CDLL(LIB_PATH)

# pda_dtype / pda_status / pda_variant
F32, BF16, FP8_E4M3 = 0, 1, 2
OK, EINVAL, EUNSUPPORTED, EHIP, ENOMEM = 0, -1, -2, -3, -4
VARIANT_AUTO, VARIANT_VECTOR, VARIANT_MFMA = 0, 1, 2
_VARIANTS = {"auto": VARIANT_AUTO, "vector": VARIANT_VECTOR, "mfma": VARIANT_MFMA}
STATUS_LEN_CLAMPED, STATUS_BAD_BLOCK, STATUS_PREFIX_SHORTENED, STATUS_BAD_OFFSETS = 1, 2, 4, 8
STATUS_HALF_RANGE = 16
NOALLOC_SCRATCH_BYTES = 32 << 20   # PDA_NOALLOC_SCRATCH_BYTES


class Problem(ctypes.Structure):
    _fields_ = [
        ("num_seqs", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("max_blocks_per_seq", ctypes.c_int32),
        ("num_blocks", ctypes.c_int64),
        ("max_seq_len", ctypes.c_int32),
        ("q_dtype", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
        ("out_dtype", ctypes.c_int32),
        ("q_tokens", ctypes.c_int32),
    ]


class Options(ctypes.Structure):
    _fields_ = [
        ("variant", ctypes.c_int32),
        ("waves_per_cu", ctypes.c_int32),
        ("min_blocks_per_wave", ctypes.c_int32),
        ("chunks_per_wave", ctypes.c_int32),
        ("min_blocks_per_chunk", ctypes.c_int32),
    ]


class PlanInfo(ctypes.Structure):
    _fields_ = [
        ("variant", ctypes.c_int32),
        ("waves", ctypes.c_int32),
        ("group_size", ctypes.c_int32),
        ("chunks_max", ctypes.c_int32),
        ("workspace_bytes", ctypes.c_int64),
    ]


class AppendProblem(ctypes.Structure):
    _fields_ = [
        ("num_seqs", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("max_blocks_per_seq", ctypes.c_int32),
        ("num_blocks", ctypes.c_int64),
        ("new_dtype", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
    ]


class PrefillProblem(ctypes.Structure):
    _fields_ = [
        ("num_seqs", ctypes.c_int32),
        ("num_tokens", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("max_blocks_per_seq", ctypes.c_int32),
        ("num_blocks", ctypes.c_int64),
        ("max_seq_len", ctypes.c_int32),
        ("q_dtype", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
        ("out_dtype", ctypes.c_int32),
    ]


_vp = ctypes.c_void_p
_lib.pda_paged_decode_attention.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_float,
                                            ctypes.POINTER(Problem), ctypes.POINTER(Options), _vp]
_lib.pda_paged_decode_attention.restype = ctypes.c_int
_lib.pda_paged_decode_attention_noalloc.argtypes = _lib.pda_paged_decode_attention.argtypes
_lib.pda_paged_decode_attention_noalloc.restype = ctypes.c_int
_lib.pda_query_plan.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(Options), ctypes.c_float,
                                ctypes.c_int32, ctypes.POINTER(PlanInfo)]
_lib.pda_query_plan.restype = ctypes.c_int
_lib.pda_paged_decode_attention_shared_prefix.argtypes = [
    _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_float, ctypes.c_int32, _vp,
    ctypes.POINTER(Problem), ctypes.POINTER(Options), _vp]
_lib.pda_paged_decode_attention_shared_prefix.restype = ctypes.c_int
_lib.pda_query_plan_shared_prefix.argtypes = [ctypes.POINTER(Problem), ctypes.POINTER(Options), ctypes.c_float,
                                              ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(PlanInfo)]
_lib.pda_query_plan_shared_prefix.restype = ctypes.c_int
_lib.pda_paged_kv_append.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.POINTER(AppendProblem), _vp]
_lib.pda_paged_kv_append.restype = ctypes.c_int
_lib.pda_paged_prefill_attention.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_float,
                                             ctypes.POINTER(PrefillProblem), _vp]
_lib.pda_paged_prefill_attention.restype = ctypes.c_int
_lib.pda_read_device_status.argtypes = [_vp]
_lib.pda_read_device_status.restype = ctypes.c_int
_lib.pda_release_workspaces.argtypes = []
_lib.pda_release_workspaces.restype = ctypes.c_int
_lib.pda_last_error.argtypes = []
_lib.pda_last_error.restype = ctypes.c_char_p
_lib.pda_version.argtypes = []
_lib.pda_version.restype = ctypes.c_int


class PdaError(RuntimeError):
    def __init__(self, code, message):
        super().__init__(f"pda error {code}: {message}")
        self.code = code


def last_error() -> str:
    return (_lib.pda_last_error() or b"").decode()


def version() -> int:
    return _lib.pda_version()


def header_symbols():
    """Names of the functions include/pda.h declares."""
    text = open(HEADER_PATH).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(pda_\w+)\s*\(", text, re.M)))


def _check(rc):
    if rc != OK:
        raise PdaError(rc, last_error())
    return rc


def make_options(variant="auto", waves_per_cu=0, min_blocks_per_wave=0, chunks_per_wave=0,
                 min_blocks_per_chunk=0) -> Options:
    v = _VARIANTS[variant] if isinstance(variant, str) else int(variant)
    return Options(v, int(waves_per_cu), int(min_blocks_per_wave), int(chunks_per_wave),
                   int(min_blocks_per_chunk))


def raw_call(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, softmax_scale,
             problem: Problem, options: Options | None = None, stream=None) -> int:
    """pda_paged_decode_attention with integer pointers; returns the status code."""
    return _lib.pda_paged_decode_attention(
        q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, ctypes.c_float(softmax_scale),
        ctypes.byref(problem), ctypes.byref(options) if options is not None else None, stream)


def raw_call_noalloc(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, softmax_scale,
                     problem: Problem, options: Options | None = None, stream=None) -> int:
    """pda_paged_decode_attention_noalloc with integer pointers; returns the status code."""
    return _lib.pda_paged_decode_attention_noalloc(
        q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, ctypes.c_float(softmax_scale),
        ctypes.byref(problem), ctypes.byref(options) if options is not None else None, stream)


def raw_call_shared_prefix(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, softmax_scale,
                           group_size, shared_blocks, problem: Problem, options: Options | None = None,
                           stream=None) -> int:
    """pda_paged_decode_attention_shared_prefix with integer pointers; returns the status code."""
    return _lib.pda_paged_decode_attention_shared_prefix(
        q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, ctypes.c_float(softmax_scale),
        int(group_size), shared_blocks, ctypes.byref(problem),
        ctypes.byref(options) if options is not None else None, stream)


def raw_kv_append(k_new, v_new, k_cache, v_cache, kv_scales, block_table, positions, problem: AppendProblem,
                  stream=None) -> int:
    """pda_paged_kv_append with integer pointers; returns the status code."""
    return _lib.pda_paged_kv_append(k_new, v_new, k_cache, v_cache, kv_scales, block_table, positions,
                                    ctypes.byref(problem), stream)


def raw_prefill(q, q_offsets, k_cache, v_cache, block_table, seq_lens, kv_scales, out, softmax_scale,
                problem: PrefillProblem, stream=None) -> int:
    """pda_paged_prefill_attention with integer pointers; returns the status code."""
    return _lib.pda_paged_prefill_attention(q, q_offsets, k_cache, v_cache, block_table, seq_lens, kv_scales, out,
                                            ctypes.c_float(softmax_scale), ctypes.byref(problem), stream)


def query_plan_shared_prefix(problem: Problem, group_size: int, options: Options | None = None,
                             softmax_scale: float = 1.0, num_compute_units: int = 256) -> PlanInfo:
    info = PlanInfo()
    _check(_lib.pda_query_plan_shared_prefix(ctypes.byref(problem),
                                             ctypes.byref(options) if options is not None else None,
                                             ctypes.c_float(softmax_scale), int(group_size),
                                             int(num_compute_units), ctypes.byref(info)))
    return info


def query_plan(problem: Problem, options: Options | None = None, softmax_scale: float = 1.0,
               num_compute_units: int = 256) -> PlanInfo:
    info = PlanInfo()
    _check(_lib.pda_query_plan(ctypes.byref(problem),
                               ctypes.byref(options) if options is not None else None,
                               ctypes.c_float(softmax_scale), int(num_compute_units), ctypes.byref(info)))
    return info


# ------------------------------------------------------------------ torch front end

def _torch():
    import torch  # noqa: WPS433 - imported lazily: the ABI tests run without it
    return torch


def _dtype_code(t, what):
    torch = _torch()
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype in (torch.uint8, torch.float8_e4m3fn):
        return FP8_E4M3
    raise TypeError(f"{what}: unsupported dtype {t.dtype}")


def _stream_handle(stream, device):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return ctypes.c_void_p(stream.cuda_stream)


def problem_for(q, k_cache, v_cache, block_table, seq_lens, max_seq_len=0, out=None) -> Problem:
    """Problem descriptor from tensor shapes and dtypes (checks they agree).
    q is [num_seqs, num_q_heads, head_dim], or [num_seqs, q_tokens, num_q_heads,
    head_dim] for several query tokens per sequence."""
    if q.dim() == 4:
        B, ntok, hq, d = q.shape
    elif q.dim() == 3:
        (B, hq, d), ntok = q.shape, 1
    else:
        raise ValueError("q must be [num_seqs, num_q_heads, head_dim] or [num_seqs, q_tokens, num_q_heads, head_dim]")
    if k_cache.dim() != 4 or v_cache.dim() != 4:
        raise ValueError("k_cache must be [NB, Hkv, 16, D] and v_cache [NB, Hkv, D, 16]")
    nb, hkv, bs, dk = k_cache.shape
    if tuple(v_cache.shape) != (nb, hkv, dk, bs):
        raise ValueError(f"v_cache shape {tuple(v_cache.shape)} != {(nb, hkv, dk, bs)} (dim-major tiles)")
    if dk != d:
        raise ValueError(f"head_dim mismatch: q {d}, cache {dk}")
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError("block_table must be [num_seqs, max_blocks_per_seq]")
    if seq_lens.shape != (B,):
        raise ValueError("seq_lens must be [num_seqs]")
    kv_dt = _dtype_code(k_cache, "k_cache")
    if _dtype_code(v_cache, "v_cache") != kv_dt:
        raise TypeError("k_cache and v_cache dtypes differ")
    q_dt = _dtype_code(q, "q")
    out_dt = _dtype_code(out, "out") if out is not None else q_dt
    return Problem(B, hq, hkv, d, bs, block_table.shape[1], nb, int(max_seq_len), q_dt, kv_dt, out_dt, ntok)


def paged_decode_attention(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out,
                           softmax_scale, max_seq_len=0, stream=None, variant="auto",
                           waves_per_cu=0, min_blocks_per_wave=0, chunks_per_wave=0,
                           min_blocks_per_chunk=0):
    """Enqueue one decode-attention step on ``stream`` (default: torch's current stream).

    All tensors live on the same HIP device and are contiguous; layouts and
    dtypes are those of include/pda.h (k_cache [NB, Hkv, 16, D], v_cache
    [NB, Hkv, D, 16], fp8 caches as uint8 or float8_e4m3fn codes plus
    kv_scales [2, NB, Hkv] fp32). ``out`` has q's shape and q's dtype or float32.
    """
    torch = _torch()
    prob, opts = _prepare(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, max_seq_len,
                          variant, waves_per_cu, min_blocks_per_wave, chunks_per_wave, min_blocks_per_chunk)
    with torch.cuda.device(q.device):
        rc = raw_call(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(),
                      seq_lens.data_ptr(), kv_scales.data_ptr() if kv_scales is not None else None,
                      out.data_ptr(), float(softmax_scale), prob, opts, _stream_handle(stream, q.device))
    _check(rc)
    return out


def paged_decode_attention_noalloc(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out,
                                   softmax_scale, max_seq_len=0, stream=None, variant="auto",
                                   waves_per_cu=0, min_blocks_per_wave=0, chunks_per_wave=0,
                                   min_blocks_per_chunk=0):
    """paged_decode_attention through the entry point that allocates nothing:
    its workspace is the library's fixed per-device scratch array
    (NOALLOC_SCRATCH_BYTES), shared by every call on the device."""
    torch = _torch()
    prob, opts = _prepare(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, max_seq_len,
                          variant, waves_per_cu, min_blocks_per_wave, chunks_per_wave, min_blocks_per_chunk)
    with torch.cuda.device(q.device):
        rc = raw_call_noalloc(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(),
                              seq_lens.data_ptr(), kv_scales.data_ptr() if kv_scales is not None else None,
                              out.data_ptr(), float(softmax_scale), prob, opts, _stream_handle(stream, q.device))
    _check(rc)
    return out


def paged_decode_attention_shared_prefix(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out,
                                         softmax_scale, group_size, shared_blocks, max_seq_len=0, stream=None,
                                         variant="auto", waves_per_cu=0, min_blocks_per_wave=0,
                                         chunks_per_wave=0, min_blocks_per_chunk=0):
    """The same step for groups of ``group_size`` consecutive sequences whose
    block tables share leading blocks; ``shared_blocks`` is an int32 device
    tensor [num_seqs / group_size] bounding each group's shared blocks (the
    library checks the bound against the block tables)."""
    torch = _torch()
    prob, opts = _prepare(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, max_seq_len,
                          variant, waves_per_cu, min_blocks_per_wave, chunks_per_wave, min_blocks_per_chunk)
    if shared_blocks.device != q.device or not shared_blocks.is_contiguous() or shared_blocks.dtype != torch.int32:
        raise ValueError(f"shared_blocks must be a contiguous int32 tensor on {q.device}")
    if group_size < 1 or q.shape[0] % group_size or shared_blocks.numel() != q.shape[0] // group_size:
        raise ValueError("shared_blocks must have num_seqs / group_size entries")
    with torch.cuda.device(q.device):
        rc = raw_call_shared_prefix(q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), block_table.data_ptr(),
                                    seq_lens.data_ptr(), kv_scales.data_ptr() if kv_scales is not None else None,
                                    out.data_ptr(), float(softmax_scale), group_size, shared_blocks.data_ptr(),
                                    prob, opts, _stream_handle(stream, q.device))
    _check(rc)
    return out


def _prepare(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, max_seq_len, variant, waves_per_cu,
             min_blocks_per_wave, chunks_per_wave, min_blocks_per_chunk):
    torch = _torch()
    tensors = {"q": q, "k_cache": k_cache, "v_cache": v_cache, "block_table": block_table,
               "seq_lens": seq_lens, "out": out}
    if kv_scales is not None:
        tensors["kv_scales"] = kv_scales
    dev = q.device
    for name, t in tensors.items():
        if not t.is_cuda or t.device != dev:
            raise ValueError(f"{name} must be on {dev}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if block_table.dtype != torch.int32 or seq_lens.dtype != torch.int32:
        raise TypeError("block_table and seq_lens must be int32")
    if kv_scales is not None and kv_scales.dtype != torch.float32:
        raise TypeError("kv_scales must be float32")
    if out.shape != q.shape or out.dtype not in (q.dtype, torch.float32):
        raise ValueError("out must have q's shape, and q's dtype or float32")
    prob = problem_for(q, k_cache, v_cache, block_table, seq_lens, max_seq_len, out)
    if kv_scales is not None and tuple(kv_scales.shape) != (2, prob.num_blocks, prob.num_kv_heads):
        raise ValueError("kv_scales must be [2, num_blocks, num_kv_heads]")
    opts = make_options(variant, waves_per_cu, min_blocks_per_wave, chunks_per_wave, min_blocks_per_chunk)
    return prob, opts


def paged_kv_append(k_new, v_new, k_cache, v_cache, kv_scales, block_table, positions, stream=None):
    """Enqueue the write of one decode step's new keys / values ([B, Hkv, D],
    float32 or bfloat16) into the paged cache at ``positions`` (int32 [B]);
    layouts as for paged_decode_attention. fp8 caches update ``kv_scales``."""
    torch = _torch()
    # Shapes first: the kernel reads block_table[b, :] for every b < B, so a
    # table with fewer rows (or a flat one) would be read past its end.
    if k_new.dim() != 3 or v_new.shape != k_new.shape or v_new.dtype != k_new.dtype:
        raise ValueError("k_new and v_new must both be [B, Hkv, D] with one dtype")
    B, hkv, d = k_new.shape
    if k_cache.dim() != 4 or v_cache.dim() != 4:
        raise ValueError("k_cache must be [NB, Hkv, 16, D] and v_cache [NB, Hkv, D, 16]")
    nb, hkv2, bs, d2 = k_cache.shape
    if (hkv2, d2) != (hkv, d) or tuple(v_cache.shape) != (nb, hkv, d, bs) or tuple(positions.shape) != (B,):
        raise ValueError("shapes: k_cache [NB, Hkv, 16, D], v_cache [NB, Hkv, D, 16], positions [B]")
    if block_table.dim() != 2 or block_table.shape[0] != B:
        raise ValueError(f"block_table must be [B, max_blocks_per_seq] with B = {B} rows (one per new token), "
                         f"got {tuple(block_table.shape)}")
    tensors = {"k_new": k_new, "v_new": v_new, "k_cache": k_cache, "v_cache": v_cache,
               "block_table": block_table, "positions": positions}
    if kv_scales is not None:
        tensors["kv_scales"] = kv_scales
    dev = k_new.device
    for name, t in tensors.items():
        if not t.is_cuda or t.device != dev:
            raise ValueError(f"{name} must be on {dev}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if block_table.dtype != torch.int32 or positions.dtype != torch.int32:
        raise TypeError("block_table and positions must be int32")
    kv_dt = _dtype_code(k_cache, "k_cache")
    if kv_dt == FP8_E4M3 and (kv_scales is None or tuple(kv_scales.shape) != (2, nb, hkv)
                              or kv_scales.dtype != torch.float32):
        raise ValueError("an fp8 cache needs float32 kv_scales [2, num_blocks, num_kv_heads]")
    prob = AppendProblem(B, hkv, d, bs, block_table.shape[1], nb, _dtype_code(k_new, "k_new"), kv_dt)
    with torch.cuda.device(dev):
        rc = raw_kv_append(k_new.data_ptr(), v_new.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                           kv_scales.data_ptr() if kv_scales is not None else None, block_table.data_ptr(),
                           positions.data_ptr(), prob, _stream_handle(stream, dev))
    _check(rc)


def paged_prefill_attention(q, q_offsets, k_cache, v_cache, block_table, seq_lens, kv_scales, out,
                            softmax_scale, max_seq_len=0, stream=None):
    """Enqueue the causal attention of packed query tokens over the paged cache.

    q and out are [T, Hq, D] (q bfloat16; out bfloat16 or float32); rows
    q_offsets[b] .. q_offsets[b + 1] - 1 (int32 [B + 1]) are the last tokens of
    sequence b, whose cache holds seq_lens[b] tokens; cache layouts as for
    paged_decode_attention. The call converts the cache tiles it reads into an
    image in the stream's workspace (V as fp16, an fp8 cache's K as bf16;
    NB * Hkv * 16 * D * 2 bytes, twice that for fp8) unless that exceeds
    PDA_PREFILL_IMAGE_MAX_MB (default 8192), in which case the kernel converts
    tiles in registers; the results are the same bit for bit.
    """
    torch = _torch()
    tensors = {"q": q, "q_offsets": q_offsets, "k_cache": k_cache, "v_cache": v_cache,
               "block_table": block_table, "seq_lens": seq_lens, "out": out}
    if kv_scales is not None:
        tensors["kv_scales"] = kv_scales
    dev = q.device
    for name, t in tensors.items():
        if not t.is_cuda or t.device != dev:
            raise ValueError(f"{name} must be on {dev}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if q.dim() != 3:
        raise ValueError("q must be [num_tokens, num_q_heads, head_dim]")
    T, hq, d = q.shape
    if k_cache.dim() != 4 or v_cache.dim() != 4:
        raise ValueError("k_cache must be [NB, Hkv, 16, D] and v_cache [NB, Hkv, D, 16]")
    nb, hkv, bs, dk = k_cache.shape
    if tuple(v_cache.shape) != (nb, hkv, dk, bs) or dk != d:
        raise ValueError("cache shapes must be k [NB, Hkv, 16, D], v [NB, Hkv, D, 16] with q's D")
    if block_table.dim() != 2 or seq_lens.dim() != 1 or block_table.shape[0] != seq_lens.shape[0]:
        raise ValueError("block_table must be [num_seqs, max_blocks_per_seq] and seq_lens [num_seqs]")
    B = seq_lens.shape[0]
    if q_offsets.shape != (B + 1,):
        raise ValueError("q_offsets must be [num_seqs + 1]")
    if any(t.dtype != torch.int32 for t in (q_offsets, block_table, seq_lens)):
        raise TypeError("q_offsets, block_table and seq_lens must be int32")
    if out.shape != q.shape:
        raise ValueError("out must have q's shape")
    kv_dt = _dtype_code(k_cache, "k_cache")
    if _dtype_code(v_cache, "v_cache") != kv_dt:
        raise TypeError("k_cache and v_cache dtypes differ")
    if kv_scales is not None and (tuple(kv_scales.shape) != (2, nb, hkv) or kv_scales.dtype != torch.float32):
        raise ValueError("kv_scales must be float32 [2, num_blocks, num_kv_heads]")
    prob = PrefillProblem(B, T, hq, hkv, d, bs, block_table.shape[1], nb, int(max_seq_len),
                          _dtype_code(q, "q"), kv_dt, _dtype_code(out, "out"))
    with torch.cuda.device(dev):
        rc = raw_prefill(q.data_ptr(), q_offsets.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                         block_table.data_ptr(), seq_lens.data_ptr(),
                         kv_scales.data_ptr() if kv_scales is not None else None, out.data_ptr(),
                         float(softmax_scale), prob, _stream_handle(stream, dev))
    _check(rc)
    return out


def read_device_status(stream=None, device=None) -> int:
    torch = _torch()
    device = device if device is not None else torch.cuda.current_device()
    with torch.cuda.device(device):
        rc = _lib.pda_read_device_status(_stream_handle(stream, device))
    if rc < 0:
        raise PdaError(rc, last_error())
    return rc


def release_workspaces() -> None:
    _check(_lib.pda_release_workspaces())
